"""Multi-hop chain oracles, in double precision (test infrastructure only).

The multi-hop KBQA model of Sec. 3.2 chains follow steps,
x^t = follow(x^{t-1}, r^t) for t = 1..T, then takes a softmax of x^T and a
cross-entropy loss against the target answer set written as a uniform
distribution over its members.  Here the relation sets are r^t = softmax(rho^t)
over relations, and each hop's output is L1-normalised, x^t = u^t / sum(u^t),
so the entity weights stay a distribution from hop to hop.  The loss is summed
over entities and averaged over the b examples.

Backward (chain rule, all in double):
  dz      = (softmax(x^T) - target) / b             (target rows sum to 1)
  du^t    = (dx^t - <dx^t, x^t>) / sum(u^t)          (per example)
  dx^{t-1}, dr^t = follow gradients at (x^{t-1}, r^t) with upstream du^t
  drho^t  = r^t * (dr^t - <dr^t, r^t>)
"""
from __future__ import annotations

import numpy as np

from . import follow_f64, follow_backward_f64


def softmax(z):
    z = np.asarray(z, np.float64)
    e = np.exp(z - z.max(axis=1, keepdims=True))
    return e / e.sum(axis=1, keepdims=True)


def chain_forward(kb_arrays, n_entities, n_relations, x0, rho):
    subj, rel, obj = kb_arrays
    xs = [np.asarray(x0, np.float64)]
    rs, sums = [], []
    for t in range(len(rho)):
        r = softmax(rho[t])
        u = follow_f64(subj, rel, obj, n_entities, n_relations, xs[-1], r)
        s = u.sum(axis=1, keepdims=True)
        if np.any(s <= 0):
            raise ValueError("a hop produced an empty entity set")
        rs.append(r)
        sums.append(s)
        xs.append(u / s)
    return xs, rs, sums


def chain_loss(kb_arrays, n_entities, n_relations, x0, rho, target):
    xs, _, _ = chain_forward(kb_arrays, n_entities, n_relations, x0, rho)
    z = xs[-1]
    zmax = z.max(axis=1, keepdims=True)
    logp = z - zmax - np.log(np.exp(z - zmax).sum(axis=1, keepdims=True))
    return float(-(np.asarray(target, np.float64) * logp).sum() / z.shape[0])


def chain_grad(kb_arrays, n_entities, n_relations, x0, rho, target):
    """Returns (loss, dx0 [b][N_E], [drho^1..drho^T] each [b][N_R])."""
    subj, rel, obj = kb_arrays
    xs, rs, sums = chain_forward(kb_arrays, n_entities, n_relations, x0, rho)
    b = xs[0].shape[0]
    target = np.asarray(target, np.float64)
    p = softmax(xs[-1])
    loss = chain_loss(kb_arrays, n_entities, n_relations, x0, rho, target)
    dx = (p - target) / b
    drho = [None] * len(rho)
    for t in range(len(rho), 0, -1):
        x_t = xs[t]
        du = (dx - (dx * x_t).sum(axis=1, keepdims=True)) / sums[t - 1]
        dxp, dr = follow_backward_f64(subj, rel, obj, n_entities, n_relations, xs[t - 1],
                                      rs[t - 1], du)
        r = rs[t - 1]
        drho[t - 1] = r * (dr - (dr * r).sum(axis=1, keepdims=True))
        dx = dxp
    return loss, dx, drho


# ---------------------------------------------------------------------------
# Residual chains of the KB-completion model (Sec. 3.2, App. E):
#   x^t = follow(x^{t-1}, r^t) + x^{t-1},  t = 1..T.
# Backward for a loss with upstream G = dL/dx^T (chain rule):
#   dx^T = G;  dr^t = follow's dR at (x^{t-1}, r^t) with upstream dx^t;
#   dx^{t-1} = follow's dX at r^t with upstream dx^t, plus dx^t.
# ---------------------------------------------------------------------------

def residual_chain(kb_arrays, n_entities, n_relations, x0, rs, weight=None):
    """[x^0, x^1, ..., x^T] for relation sets rs = [r^1..r^T] (each [b][N_R])."""
    subj, rel, obj = kb_arrays
    xs = [np.asarray(x0, np.float64)]
    for r in rs:
        xs.append(follow_f64(subj, rel, obj, n_entities, n_relations, xs[-1], r, weight) + xs[-1])
    return xs


def residual_chain_grad(kb_arrays, n_entities, n_relations, x0, rs, G, weight=None):
    """(dL/dx^0, [dL/dr^1..dL/dr^T]) for upstream G = dL/dx^T."""
    subj, rel, obj = kb_arrays
    xs = residual_chain(kb_arrays, n_entities, n_relations, x0, rs, weight)
    dx = np.asarray(G, np.float64)
    drs = [None] * len(rs)
    for t in range(len(rs), 0, -1):
        dxp, dr = follow_backward_f64(subj, rel, obj, n_entities, n_relations, xs[t - 1],
                                      rs[t - 1], dx, weight)
        drs[t - 1] = dr
        dx = dxp + dx
    return dx, drs
