"""Seeded synthetic knowledge bases and inputs for relation-set following.

This module only draws random numbers and shapes them into the workloads the
tests and the benchmark use; it holds none of the follow arithmetic.  Both the
CPU oracle and the HIP path consume exactly these arrays.

Workloads (five shapes; each may be scaled down for fast tests):

* ``tiny``    -- uniform triples, k-hot X, one-hot R, dY = 1 (integer valued).
* ``metaqa``  -- a MetaQA-shaped KB (about 43 k entities, 9 relations plus their
  inverses, Zipf subject out-degree), dense softmax X and R (Sec. 3.2, KBQA).
* ``chain3``  -- the tiny KB driven through a three-hop chain
  x^t = follow(x^{t-1}, r^t) with a cross-entropy loss at the end (Sec. 3.2).
* ``large``   -- 10 M entities / 50 M triples / 600 relations with Zipf
  subject, object and relation marginals (the scale of the Freebase subset used
  for WebQuestionsSP, Sec. 3.2), 1 %-dense X.
* ``train``   -- 2 M entities / 20 M triples / 1000 relations, Zipf subjects
  with heavy hubs, b = 256.

Conventions: ids are 0-based (the paper numbers entities from 1, Sec. 2.1).
Activations are returned in the paper's batch-major orientation, ``[b][N]``
(row beta is example beta, Sec. 2.3 and App. C); callers that want the
entity-major ``[N][b]`` layout transpose.

Zipf(s) over N items means the truncated rank-frequency law p_k ~ k^-s,
k = 1..N, mapped to ids through a seeded permutation per role.  Distinct
triples are obtained by redrawing the deficit until exactly N_T distinct
(s, r, o) remain; the returned order is a seeded shuffle.
"""
from __future__ import annotations

import dataclasses
import hashlib

import numpy as np
from concurrent.futures import ThreadPoolExecutor

ROOT_SEED = 20020615

# RNG streams (one independent generator per purpose).
ST_TRIPLES, ST_X, ST_R, ST_DY, ST_TARGET, ST_PERM = 0, 1, 2, 3, 4, 5


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    index: int              # position in the workload list; part of every seed
    n_entities: int
    n_relations: int
    n_triples: int
    batch: int
    subj_law: tuple         # ("uniform",) or ("zipf", s)
    obj_law: tuple
    rel_law: tuple
    inverse_pairs: bool = False   # metaqa: half base triples, half (o, r + N_R/2, s)
    x_kind: str = "khot"          # khot | softmax | sparse1pct | seed1
    r_kind: str = "onehot"        # onehot | softmax1 | softmax2
    dy_kind: str = "ones"         # ones | normal | ce
    scale_tag: int = 0            # 0 = full size; scaled variants get their own seeds
    kb_source: str = ""           # draw the triples of another workload (chain3 uses tiny's KB)

    def scaled(self, n_entities, n_triples, batch=None, n_relations=None, tag=1):
        return dataclasses.replace(
            self, n_entities=int(n_entities), n_triples=int(n_triples),
            batch=int(self.batch if batch is None else batch),
            n_relations=int(self.n_relations if n_relations is None else n_relations),
            scale_tag=int(tag))

    @property
    def label(self):
        s = f"{self.name}(NE={self.n_entities},NR={self.n_relations},NT={self.n_triples},b={self.batch})"
        return s


TINY = Workload("tiny", 0, 1_000, 10, 5_000, 4, ("uniform",), ("uniform",), ("uniform",),
                x_kind="khot", r_kind="onehot", dy_kind="ones")
METAQA = Workload("metaqa", 1, 43_000, 18, 190_000, 128, ("zipf", 1.1), ("uniform",), ("uniform",),
                  inverse_pairs=True, x_kind="softmax", r_kind="softmax1", dy_kind="normal")
CHAIN3 = Workload("chain3", 2, 1_000, 10, 5_000, 256, ("uniform",), ("uniform",), ("uniform",),
                  x_kind="seed1", r_kind="softmax1", dy_kind="ce", kb_source="tiny")
LARGE = Workload("large", 3, 10_000_000, 600, 50_000_000, 32, ("zipf", 1.05), ("zipf", 1.05),
                 ("zipf", 1.2), x_kind="sparse1pct", r_kind="softmax2", dy_kind="normal")
TRAIN = Workload("train", 4, 2_000_000, 1_000, 20_000_000, 256, ("zipf", 1.1), ("uniform",),
                 ("uniform",), x_kind="softmax", r_kind="softmax1", dy_kind="normal")

WORKLOADS = {w.name: w for w in (TINY, METAQA, CHAIN3, LARGE, TRAIN)}


def rng(w: Workload, stream: int, sub: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([ROOT_SEED, w.index, stream, w.scale_tag, sub])))


# ----------------------------------------------------------------------------
# triples
# ----------------------------------------------------------------------------

def _law_probs(law, n):
    if law[0] == "uniform":
        return None
    s = float(law[1])
    p = np.arange(1, n + 1, dtype=np.float64) ** (-s)
    return p / p.sum()


def _draw_role(g, law, n, count, perm, shuffle=True):
    """``count`` iid ids from ``law`` over ``n`` items (random order unless shuffle=False)."""
    p = _law_probs(law, n)
    if p is None:
        return g.integers(0, n, size=count, dtype=np.int32)
    counts = g.multinomial(count, p)
    ranks = np.repeat(np.arange(n, dtype=np.int32), counts)
    if shuffle:
        g.shuffle(ranks)
    return perm[ranks]


def _distinct_triples(w: Workload, n_e, n_r, n_t, subj_law, obj_law, rel_law, sub=0):
    gp = rng(w, ST_PERM, sub)
    perm_s = gp.permutation(n_e).astype(np.int32)
    perm_o = gp.permutation(n_e).astype(np.int32)
    perm_r = gp.permutation(n_r).astype(np.int32)
    NE, NR = np.uint64(n_e), np.uint64(n_r)
    draws = [0]

    def draw(count):
        # Each role has its own generator, so the three draws run in parallel.
        # The subject ids stay grouped by rank: pairing them with independently
        # shuffled relation and object ids still gives iid (s, r, o) triples.
        k = draws[0]
        draws[0] += 1
        jobs = [(subj_law, n_e, perm_s, False), (rel_law, n_r, perm_r, True),
                (obj_law, n_e, perm_o, True)]
        def one(j):
            law, n, perm, shuf = jobs[j]
            g = rng(w, ST_TRIPLES, sub * 1000003 + k * 3 + j)
            return _draw_role(g, law, n, count, perm, shuf).astype(np.uint64)
        with ThreadPoolExecutor(3) as ex:
            s, r, o = ex.map(one, range(3))
        return (s * NR + r) * NE + o

    if n_t > n_e * n_e * n_r:
        raise ValueError("more distinct triples requested than exist")
    keys = np.unique(draw(n_t)) if n_t else np.zeros(0, np.uint64)
    g = rng(w, ST_TRIPLES, sub * 1000003 + 999_999)
    rate = max(len(keys) / max(n_t, 1), 0.05)
    rounds = 0
    while len(keys) < n_t:
        rounds += 1
        if rounds > 200:
            raise RuntimeError("could not draw enough distinct triples")
        deficit = n_t - len(keys)
        m = int(deficit / rate * 1.25) + 1024
        u2 = np.unique(draw(m))
        pos = np.minimum(np.searchsorted(keys, u2), max(len(keys) - 1, 0))
        fresh = (keys[pos] != u2) if len(keys) else np.ones(len(u2), bool)
        new = u2[fresh]
        rate = max(len(new) / m, 0.01)
        if len(new) > deficit:
            new = np.sort(new[g.choice(len(new), size=deficit, replace=False)])
        keys = np.sort(np.concatenate([keys, new]))
    keys = keys[g.permutation(n_t)]
    o = (keys % NE).astype(np.int32)
    t = keys // NE
    r = (t % NR).astype(np.int32)
    s = (t // NR).astype(np.int32)
    return s, r, o


@dataclasses.dataclass
class KB:
    workload: Workload
    subj: np.ndarray   # int32 [N_T], caller order
    rel: np.ndarray
    obj: np.ndarray

    @property
    def n_entities(self):
        return self.workload.n_entities

    @property
    def n_relations(self):
        return self.workload.n_relations

    @property
    def n_triples(self):
        return int(self.subj.shape[0])

    def sha256(self):
        h = hashlib.sha256()
        for a in (self.subj, self.rel, self.obj):
            h.update(np.ascontiguousarray(a).tobytes())
        return h.hexdigest()

    def stats(self):
        ne, nr = self.n_entities, self.n_relations
        out_deg = np.bincount(self.subj, minlength=ne)
        in_deg = np.bincount(self.obj, minlength=ne)
        rel_seg = np.bincount(self.rel, minlength=nr)
        return {
            "max_out_degree": int(out_deg.max(initial=0)),
            "max_in_degree": int(in_deg.max(initial=0)),
            "zero_out_degree": int((out_deg == 0).sum()),
            "zero_in_degree": int((in_deg == 0).sum()),
            "subjects_deg_ge_1e4": int((out_deg >= 10_000).sum()),
            "objects_deg_ge_1e4": int((in_deg >= 10_000).sum()),
            "max_rel_segment": int(rel_seg.max(initial=0)),
        }


def make_kb(w: Workload) -> KB:
    """The workload's triple store, in the caller order the library receives."""
    if w.kb_source:
        src = dataclasses.replace(WORKLOADS[w.kb_source], n_entities=w.n_entities,
                                  n_relations=w.n_relations, n_triples=w.n_triples,
                                  scale_tag=w.scale_tag)
        kb = make_kb(src)
        return KB(w, kb.subj, kb.rel, kb.obj)
    if w.inverse_pairs:
        half_r = w.n_relations // 2
        s, r, o = _distinct_triples(w, w.n_entities, half_r, w.n_triples // 2,
                                    w.subj_law, w.obj_law, w.rel_law)
        s2 = np.concatenate([s, o])
        r2 = np.concatenate([r, r + half_r]).astype(np.int32)
        o2 = np.concatenate([o, s])
        order = rng(w, ST_TRIPLES, 7).permutation(len(s2))
        return KB(w, s2[order].copy(), r2[order].copy(), o2[order].copy())
    s, r, o = _distinct_triples(w, w.n_entities, w.n_relations, w.n_triples,
                                w.subj_law, w.obj_law, w.rel_law)
    return KB(w, s, r, o)


def kb_from_arrays(w: Workload, subj, rel, obj) -> KB:
    return KB(w, np.ascontiguousarray(subj, np.int32), np.ascontiguousarray(rel, np.int32),
              np.ascontiguousarray(obj, np.int32))


# ----------------------------------------------------------------------------
# activations (paper orientation [b][N])
# ----------------------------------------------------------------------------

def _softmax_rows(z):
    z = z - z.max(axis=1, keepdims=True)
    e = np.exp(z)
    return e / e.sum(axis=1, keepdims=True)


def _per_row(w: Workload, stream: int, sub: int, b: int, n: int, fill):
    """[b][n] float32, row beta filled by ``fill(generator, row)`` with its own seed."""
    out = np.empty((b, n), np.float32)

    def one(beta):
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(
            [ROOT_SEED, w.index, stream, w.scale_tag, sub, beta])))
        fill(g, out[beta])

    if b * n >= 1 << 20:
        with ThreadPoolExecutor(8) as ex:
            list(ex.map(one, range(b)))
    else:
        for beta in range(b):
            one(beta)
    return out


def _fill_khot(g, row):
    row[:] = 0.0
    n = row.shape[0]
    k = int(g.integers(1, 6))
    row[g.choice(n, size=min(k, n), replace=False)] = 1.0


def _fill_softmax(g, row):
    g.standard_normal(row.shape[0], dtype=np.float32, out=row)
    row -= row.max()
    np.exp(row, out=row)
    row /= np.float32(row.sum(dtype=np.float64))


def _fill_sparse1pct(g, row):
    row[:] = 0.0
    n = row.shape[0]
    nnz = max(1, n // 100)
    cols = g.choice(n, size=nnz, replace=False)
    v = 1.0 - g.random(nnz)          # values in (0, 1]
    row[cols] = (v / v.sum()).astype(np.float32)


def _fill_normal(g, row):
    g.standard_normal(row.shape[0], dtype=np.float32, out=row)


def make_x(w: Workload, kind: str | None = None, sub: int = 0) -> np.ndarray:
    kind = kind or w.x_kind
    fill = {"khot": _fill_khot, "softmax": _fill_softmax, "sparse1pct": _fill_sparse1pct,
            "normal": _fill_normal}[kind]
    return _per_row(w, ST_X, sub, w.batch, w.n_entities, fill)


def make_r(w: Workload, kind: str | None = None, sub: int = 0) -> np.ndarray:
    kind = kind or w.r_kind
    b, n = w.batch, w.n_relations
    g = rng(w, ST_R, sub)
    if kind == "onehot":
        r = np.zeros((b, n), np.float32)
        r[np.arange(b), g.integers(0, n, size=b)] = 1.0
        return r
    if kind == "softmax1":
        return _softmax_rows(g.standard_normal((b, n))).astype(np.float32)
    if kind == "softmax2":
        return _softmax_rows(2.0 * g.standard_normal((b, n))).astype(np.float32)
    if kind == "normal":
        return g.standard_normal((b, n), dtype=np.float32)
    raise ValueError(kind)


def make_dy(w: Workload, kind: str | None = None, sub: int = 0) -> np.ndarray:
    kind = kind or w.dy_kind
    b, n = w.batch, w.n_entities
    if kind == "ones":
        return np.ones((b, n), np.float32)
    if kind == "normal":
        return _per_row(w, ST_DY, sub, b, n, _fill_normal)
    raise ValueError(kind)


def make_integer_inputs(w: Workload, sub: int = 0):
    """k-hot X, one-hot R, dY = 1 on any workload's KB (every sum stays an exact integer)."""
    return (make_x(w, "khot", sub), make_r(w, "onehot", sub), make_dy(w, "ones", sub))


# ----------------------------------------------------------------------------
# three-hop chain inputs
# ----------------------------------------------------------------------------

def _has_path(adj, start, hops):
    frontier = {start}
    for _ in range(hops):
        nxt = set()
        for e in frontier:
            nxt.update(adj.get(e, ()))
        if not nxt:
            return False
        frontier = nxt
    return True


def make_chain_inputs(w: Workload, kb: KB, hops: int = 3, sub: int = 0):
    """Seeds, relation logits and targets for the multi-hop chain.

    Returns ``(x0 [b][N_E] one-hot, rho [hops][b][N_R] N(0,1) logits,
    target [b][N_E] uniform over k ~ U{1..5} distinct entities)``.  Every seed
    starts a path of ``hops`` edges, so no hop's output row is all zero.
    """
    b, n = w.batch, w.n_entities
    adj = {}
    for s_, o_ in zip(kb.subj.tolist(), kb.obj.tolist()):
        adj.setdefault(s_, []).append(o_)
    g = rng(w, ST_X, sub)
    x0 = np.zeros((b, n), np.float32)
    for beta in range(b):
        while True:
            e = int(g.integers(0, n))
            if _has_path(adj, e, hops):
                break
        x0[beta, e] = 1.0
    gr = rng(w, ST_R, sub)
    rho = gr.standard_normal((hops, b, w.n_relations)).astype(np.float32)
    gt = rng(w, ST_TARGET, sub)
    tgt = np.zeros((b, n), np.float32)
    for beta in range(b):
        k = int(gt.integers(1, 6))
        tgt[beta, gt.choice(n, size=k, replace=False)] = 1.0 / k
    return x0, rho, tgt


# ----------------------------------------------------------------------------
# grid KB of the scalability experiment (Sec. 3.1)
# ----------------------------------------------------------------------------

GRID_INDEX = 5      # seed slot of the grid workloads


def grid_kb(n: int, n_relations: int = 4):
    """The n x n grid KB: every cell is an entity linked to its neighbours by
    north / south / east / west edges.  With n_relations = 4 the relation is
    the direction; otherwise every edge gets one of n_relations invented
    relation names uniformly at random (seeded), as in the relation sweep of
    Sec. 3.1.  Cell (a, c) is entity a * n + c.  Returns int32 (subj, rel, obj)."""
    a, c = np.meshgrid(np.arange(n), np.arange(n), indexing="ij")
    a, c = a.ravel(), c.ravel()
    subj, rel, obj = [], [], []
    for k, (da, dc) in enumerate(((-1, 0), (1, 0), (0, 1), (0, -1))):
        ok = (a + da >= 0) & (a + da < n) & (c + dc >= 0) & (c + dc < n)
        subj.append(a[ok] * n + c[ok])
        obj.append((a[ok] + da) * n + c[ok] + dc)
        rel.append(np.full(int(ok.sum()), k))
    subj, rel, obj = (np.concatenate(v).astype(np.int32) for v in (subj, rel, obj))
    if n_relations != 4:
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(
            [ROOT_SEED, GRID_INDEX, ST_TRIPLES, n, n_relations])))
        rel = g.integers(0, n_relations, len(subj)).astype(np.int32)
    return subj, rel, obj


def grid_inputs(n: int, n_relations: int, batch: int = 128):
    """One-hot random cells and relation weights 1 + U(0, 0.001) (the grid
    experiments of App. E), in batch-major [b][N] orientation."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(
        [ROOT_SEED, GRID_INDEX, ST_X, n, n_relations, batch])))
    x = np.zeros((batch, n * n), np.float32)
    x[np.arange(batch), g.integers(0, n * n, batch)] = 1.0
    r = (1.0 + 0.001 * g.random((batch, n_relations))).astype(np.float32)
    return x, r
