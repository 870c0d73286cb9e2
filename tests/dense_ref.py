"""Dense-matrix evaluations of the paper's equations, used to pin the oracle.

Every function here builds the paper's matrices explicitly (numpy float64) and
uses library matrix products; none shares code with the oracle's triple loop.

* ``reified``   -- Eq. 4 (Sec. 2.3): (X M_subj^T (.) R M_rel^T) M_obj
* ``naive``     -- Eq. 1-2 (Sec. 2.2): x M_R with M_R = sum_k r[k] M_{r_k}, per example
* ``late``      -- Eq. 3 (Sec. 2.3, App. C): sum_k R[:, k] * (X M_k)
* ``reified_grads`` -- the adjoint of Eq. 4 by matrix calculus:
  with A = X M_subj^T and B = R M_rel^T, Y = (A (.) B) M_obj, so
  dA = (dY M_obj^T) (.) B, dX = dA M_subj and dB = (dY M_obj^T) (.) A, dR = dB M_rel.
"""
import numpy as np


def matrices(subj, rel, obj, n_e, n_r, weight=None):
    n_t = len(subj)
    w = np.ones(n_t) if weight is None else np.asarray(weight, np.float64)
    Ms = np.zeros((n_t, n_e))
    Mo = np.zeros((n_t, n_e))
    Mr = np.zeros((n_t, n_r))
    Ms[np.arange(n_t), subj] = 1.0
    Mo[np.arange(n_t), obj] = 1.0
    Mr[np.arange(n_t), rel] = w          # soft KB: weight stored in M_rel (App. A)
    return Ms, Mr, Mo


def relation_matrices(subj, rel, obj, n_e, n_r, weight=None):
    """M_k[i, j] = weight of r_k(x_i, x_j) (Sec. 2.1), summed over duplicate triples."""
    w = np.ones(len(subj)) if weight is None else np.asarray(weight, np.float64)
    M = np.zeros((n_r, n_e, n_e))
    np.add.at(M, (np.asarray(rel), np.asarray(subj), np.asarray(obj)), w)
    return M


def reified(subj, rel, obj, n_e, n_r, X, R, weight=None):
    Ms, Mr, Mo = matrices(subj, rel, obj, n_e, n_r, weight)
    X = np.asarray(X, np.float64)
    R = np.asarray(R, np.float64)
    return ((X @ Ms.T) * (R @ Mr.T)) @ Mo


def naive(subj, rel, obj, n_e, n_r, X, R, weight=None):
    M = relation_matrices(subj, rel, obj, n_e, n_r, weight)
    X = np.asarray(X, np.float64)
    R = np.asarray(R, np.float64)
    out = np.zeros((X.shape[0], n_e))
    for beta in range(X.shape[0]):
        MR = np.tensordot(R[beta], M, axes=(0, 0))    # Eq. 1
        out[beta] = X[beta] @ MR                      # Eq. 2
    return out


def late(subj, rel, obj, n_e, n_r, X, R, weight=None):
    M = relation_matrices(subj, rel, obj, n_e, n_r, weight)
    X = np.asarray(X, np.float64)
    R = np.asarray(R, np.float64)
    out = np.zeros((X.shape[0], n_e))
    for k in range(n_r):
        out += R[:, k:k + 1] * (X @ M[k])             # Eq. 3
    return out


def reified_grads(subj, rel, obj, n_e, n_r, X, R, dY, weight=None):
    Ms, Mr, Mo = matrices(subj, rel, obj, n_e, n_r, weight)
    X = np.asarray(X, np.float64)
    R = np.asarray(R, np.float64)
    dY = np.asarray(dY, np.float64)
    A, B = X @ Ms.T, R @ Mr.T
    G = dY @ Mo.T
    return (G * B) @ Ms, (G * A) @ Mr
