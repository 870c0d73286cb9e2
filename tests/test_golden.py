"""Hand-worked toy example of Sec. 2.2 (see tests/golden/toy_movie_kb.txt)."""
import os

import numpy as np

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


def load_toy():
    ent, rel, facts, queries = {}, {}, [], []
    with open(os.path.join(HERE, "golden", "toy_movie_kb.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            kind, rest = line.split(" ", 1)
            if kind == "entity":
                i, name = rest.split()
                ent[name] = int(i)
            elif kind == "relation":
                i, name = rest.split()
                rel[name] = int(i)
            elif kind == "fact":
                facts.append(tuple(rest.split()))
            elif kind == "query":
                lhs, rhs = rest.split("->")
                parts = [p.strip() for p in lhs.split("|")]
                want = {}
                for tok in rhs.split():
                    name, wgt = tok.split(":")
                    want[name] = float(wgt)
                queries.append((parts[0].split(","), [p.split(",") for p in parts[1:]], want))
    return ent, rel, facts, queries


def test_toy_movie_kb_answers():
    ent, rel, facts, queries = load_toy()
    s = np.array([ent[a] for a, _, _ in facts], np.int32)
    r = np.array([rel[k] for _, k, _ in facts], np.int32)
    o = np.array([ent[c] for _, _, c in facts], np.int32)
    n_e, n_r = len(ent), len(rel)
    for seeds, hops, want in queries:
        x = np.zeros((1, n_e), np.float32)
        x[0, [ent[e] for e in seeds]] = 1.0
        for rels in hops:
            rv = np.zeros((1, n_r), np.float32)
            rv[0, [rel[k] for k in rels]] = 1.0
            x = oracle.follow(s, r, o, n_e, n_r, x, rv)
        expect = np.zeros(n_e, np.float32)
        for name, wgt in want.items():
            expect[ent[name]] = wgt
        assert np.array_equal(x[0], expect), (seeds, hops)
