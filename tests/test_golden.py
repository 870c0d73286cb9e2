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


def test_two_hop_chain_loss_closed_form():
    """A hand-worked two-hop chain of the multi-hop model (Sec. 3.2) on the
    toy KB, pinning oracle.chain's forward and loss against a closed form.

    Seed dir_q; rho^1 = log(1, 1, 2, 4) over (directed, produced, wrote,
    starring), so r^1 = (1, 1, 2, 4) / 8; rho^2 = 0, so r^2 = 1/4 each.
    Hop 1: u^1 = movie_a 1/8 (directed), movie_b 1/8 + 1/8 (directed and
    produced), movie_c 1/8 (produced), movie_d 2/8 (wrote); sum 3/4, so
    x^1 = (1/6, 1/3, 1/6, 1/3) on movies a..d.
    Hop 2 (starring only leaves the movies): u^2 = actor_u (x_a + x_d) / 4
    = 1/8, actor_v (x_a + x_b) / 4 = 1/8, actor_w x_c / 4 = 1/24; sum 7/24,
    so x^2 = (3/7, 3/7, 1/7) on actors u, v, w and 0 on the six others.
    Target uniform over {actor_u, actor_v}: softmax over the 9 entities has
    normaliser Z = 6 + 2 e^{3/7} + e^{1/7}, and the cross-entropy is
    -(1/2)(3/7 - ln Z) - (1/2)(3/7 - ln Z) = ln Z - 3/7."""
    import math
    from oracle import chain
    ent, rel, facts, _ = load_toy()
    s = np.array([ent[a] for a, _, _ in facts], np.int32)
    r = np.array([rel[k] for _, k, _ in facts], np.int32)
    o = np.array([ent[c] for _, _, c in facts], np.int32)
    n_e, n_r = len(ent), len(rel)
    x0 = np.zeros((1, n_e))
    x0[0, ent["dir_q"]] = 1.0
    order = [rel[k] for k in ("directed", "produced", "wrote", "starring")]
    rho = np.zeros((2, 1, n_r))
    rho[0, 0, order] = np.log([1.0, 1.0, 2.0, 4.0])
    target = np.zeros((1, n_e))
    target[0, [ent["actor_u"], ent["actor_v"]]] = 0.5
    xs, _, _ = chain.chain_forward((s, r, o), n_e, n_r, x0, rho)
    want1 = np.zeros(n_e)
    for name, v in (("movie_a", 1 / 6), ("movie_b", 1 / 3), ("movie_c", 1 / 6), ("movie_d", 1 / 3)):
        want1[ent[name]] = v
    want2 = np.zeros(n_e)
    for name, v in (("actor_u", 3 / 7), ("actor_v", 3 / 7), ("actor_w", 1 / 7)):
        want2[ent[name]] = v
    np.testing.assert_allclose(xs[1][0], want1, rtol=0, atol=1e-15)
    np.testing.assert_allclose(xs[2][0], want2, rtol=0, atol=1e-15)
    loss = chain.chain_loss((s, r, o), n_e, n_r, x0, rho, target)
    closed = math.log(6 + 2 * math.exp(3 / 7) + math.exp(1 / 7)) - 3 / 7
    assert abs(loss - closed) <= 1e-14, (loss, closed)
    assert abs(closed - 1.8961362) < 1e-7
    # Planted mistake: with the target on actor_w instead, the loss is
    # ln Z - 1/7, which the pin tells apart.
    t2 = np.zeros((1, n_e))
    t2[0, ent["actor_w"]] = 1.0
    assert abs(chain.chain_loss((s, r, o), n_e, n_r, x0, rho, t2) -
               (math.log(6 + 2 * math.exp(3 / 7) + math.exp(1 / 7)) - 1 / 7)) <= 1e-14
