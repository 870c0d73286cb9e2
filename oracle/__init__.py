"""CPU oracle for relation-set following (test infrastructure only).

Only the tests, ``__graft_entry__.smoke`` and the benchmark's CPU-baseline leg
use this package.  The product library never imports it, and it imports
nothing from the product.

* :func:`follow`, :func:`follow_backward`, :func:`sampled` -- the per-triple
  definition of Eq. 4 and its gradients (a C triple loop, double accumulation,
  one rounding to float), in the paper's batch-major orientation ``[b][N]``.
* :func:`follow_f64`, :func:`follow_backward_f64` -- the same sums kept in
  double, for multi-hop chains.
* :func:`follow_residual`, :func:`follow_backward_residual` -- the residual hop
  of the KB-completion chains (Sec. 3.2, App. E): follow(X, R) + gamma * X.
* :func:`follow_accumulate` -- follow(X, R) + gamma * Z for any Z (the
  residual hop with Z = X; adding into an existing output with Z = Y).
* :mod:`oracle.chain` -- the three-hop chain with its softmax, L1 normalisation
  and cross-entropy loss, and the residual chain, forward and backward, in
  double.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "kb_oracle.c")
_LIB = os.path.join(_HERE, "libkboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain -O2, no fast-math, OpenMP over examples)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                               "-Wall", "-Wextra", "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        i64, i32, p = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p
        lib.ora_follow.argtypes = [i64, i64, i64, p, p, p, p, i32, p, p, p, i32]
        lib.ora_follow_backward.argtypes = [i64, i64, i64, p, p, p, p, i32, p, p, p, p, p, i32]
        lib.ora_sampled.argtypes = [i32, i64, i64, i64, p, p, p, p, i32, p, p, p, i32, p, p, i32]
        lib.ora_follow_f64.argtypes = [i64, i64, i64, p, p, p, p, i32, p, p, p]
        lib.ora_follow_backward_f64.argtypes = [i64, i64, i64, p, p, p, p, i32, p, p, p, p, p]
        f32 = ctypes.c_float
        lib.ora_follow_residual.argtypes = [i64, i64, i64, p, p, p, p, i32, p, p, f32, p, i32]
        lib.ora_follow_backward_residual.argtypes = [i64, i64, i64, p, p, p, p, i32, p, p, p, f32,
                                                     p, p, i32]
        lib.ora_follow_accumulate.argtypes = [i64, i64, i64, p, p, p, p, i32, p, p, p, f32, p,
                                              i32]
        for f in (lib.ora_follow, lib.ora_follow_backward, lib.ora_sampled, lib.ora_follow_f64,
                  lib.ora_follow_backward_f64, lib.ora_follow_residual,
                  lib.ora_follow_backward_residual, lib.ora_follow_accumulate):
            f.restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _ids(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _f32(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float32)


def _f64(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float64)


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"oracle {what} failed with code {rc}")


def follow(subj, rel, obj, n_entities, n_relations, X, R, weight=None, nthreads=0):
    """Y[b][N_E] = follow(X, R) (Eq. 4), X [b][N_E], R [b][N_R]."""
    subj, rel, obj = _ids(subj), _ids(rel), _ids(obj)
    X, R, weight = _f32(X), _f32(R), _f32(weight)
    b = X.shape[0]
    assert X.shape == (b, n_entities) and R.shape == (b, n_relations)
    Y = np.empty((b, n_entities), np.float32)
    rc = _load().ora_follow(n_entities, n_relations, len(subj), _ptr(subj), _ptr(rel), _ptr(obj),
                            _ptr(weight), b, _ptr(X), _ptr(R), _ptr(Y), nthreads)
    _check(rc, "follow")
    return Y


def follow_backward(subj, rel, obj, n_entities, n_relations, X, R, dY, weight=None,
                    want_dx=True, want_dr=True, nthreads=0):
    """(dX [b][N_E], dR [b][N_R]) for upstream gradient dY [b][N_E]."""
    subj, rel, obj = _ids(subj), _ids(rel), _ids(obj)
    X, R, dY, weight = _f32(X), _f32(R), _f32(dY), _f32(weight)
    b = dY.shape[0]
    dX = np.empty((b, n_entities), np.float32) if want_dx else None
    dR = np.empty((b, n_relations), np.float32) if want_dr else None
    rc = _load().ora_follow_backward(n_entities, n_relations, len(subj), _ptr(subj), _ptr(rel),
                                     _ptr(obj), _ptr(weight), b, _ptr(X), _ptr(R), _ptr(dY),
                                     _ptr(dX), _ptr(dR), nthreads)
    _check(rc, "follow_backward")
    return dX, dR


SAMPLE_Y, SAMPLE_DX, SAMPLE_DR = 0, 1, 2


def sampled(which, subj, rel, obj, n_entities, n_relations, ids, X=None, R=None, dY=None,
            weight=None, nthreads=0):
    """Selected columns of Y (which=0, object ids), dX (1, subject ids) or dR (2, relation ids).

    Returns [b][len(ids)].
    """
    subj, rel, obj, ids = _ids(subj), _ids(rel), _ids(obj), _ids(ids)
    X, R, dY, weight = _f32(X), _f32(R), _f32(dY), _f32(weight)
    b = (X if X is not None else dY).shape[0]
    out = np.empty((b, len(ids)), np.float32)
    rc = _load().ora_sampled(which, n_entities, n_relations, len(subj), _ptr(subj), _ptr(rel),
                             _ptr(obj), _ptr(weight), b, _ptr(X), _ptr(R), _ptr(dY), len(ids),
                             _ptr(ids), _ptr(out), nthreads)
    _check(rc, "sampled")
    return out


def follow_f64(subj, rel, obj, n_entities, n_relations, X, R, weight=None):
    subj, rel, obj = _ids(subj), _ids(rel), _ids(obj)
    X, R, weight = _f64(X), _f64(R), _f64(weight)
    b = X.shape[0]
    Y = np.empty((b, n_entities), np.float64)
    rc = _load().ora_follow_f64(n_entities, n_relations, len(subj), _ptr(subj), _ptr(rel),
                                _ptr(obj), _ptr(weight), b, _ptr(X), _ptr(R), _ptr(Y))
    _check(rc, "follow_f64")
    return Y


def follow_backward_f64(subj, rel, obj, n_entities, n_relations, X, R, dY, weight=None):
    subj, rel, obj = _ids(subj), _ids(rel), _ids(obj)
    X, R, dY, weight = _f64(X), _f64(R), _f64(dY), _f64(weight)
    b = dY.shape[0]
    dX = np.empty((b, n_entities), np.float64)
    dR = np.empty((b, n_relations), np.float64)
    rc = _load().ora_follow_backward_f64(n_entities, n_relations, len(subj), _ptr(subj),
                                         _ptr(rel), _ptr(obj), _ptr(weight), b, _ptr(X), _ptr(R),
                                         _ptr(dY), _ptr(dX), _ptr(dR))
    _check(rc, "follow_backward_f64")
    return dX, dR


def follow_residual(subj, rel, obj, n_entities, n_relations, X, R, gamma=1.0, weight=None,
                    nthreads=0):
    """Y = follow(X, R) + gamma * X, rounded to float once."""
    subj, rel, obj = _ids(subj), _ids(rel), _ids(obj)
    X, R, weight = _f32(X), _f32(R), _f32(weight)
    b = X.shape[0]
    Y = np.empty((b, n_entities), np.float32)
    rc = _load().ora_follow_residual(n_entities, n_relations, len(subj), _ptr(subj), _ptr(rel),
                                     _ptr(obj), _ptr(weight), b, _ptr(X), _ptr(R), gamma,
                                     _ptr(Y), nthreads)
    _check(rc, "follow_residual")
    return Y


def follow_accumulate(subj, rel, obj, n_entities, n_relations, X, R, Z, gamma=1.0, weight=None,
                      nthreads=0):
    """Y = follow(X, R) + gamma * Z (Z [b][N_E], any array of Y's shape),
    rounded to float once."""
    subj, rel, obj = _ids(subj), _ids(rel), _ids(obj)
    X, R, Z, weight = _f32(X), _f32(R), _f32(Z), _f32(weight)
    b = X.shape[0]
    assert Z.shape == X.shape
    Y = np.empty((b, n_entities), np.float32)
    rc = _load().ora_follow_accumulate(n_entities, n_relations, len(subj), _ptr(subj), _ptr(rel),
                                       _ptr(obj), _ptr(weight), b, _ptr(X), _ptr(R), _ptr(Z),
                                       gamma, _ptr(Y), nthreads)
    _check(rc, "follow_accumulate")
    return Y


def follow_backward_residual(subj, rel, obj, n_entities, n_relations, X, R, dY, gamma=1.0,
                             weight=None, nthreads=0):
    """(dX, dR) of the residual hop: dX = follow's dX + gamma * dY."""
    subj, rel, obj = _ids(subj), _ids(rel), _ids(obj)
    X, R, dY, weight = _f32(X), _f32(R), _f32(dY), _f32(weight)
    b = dY.shape[0]
    dX = np.empty((b, n_entities), np.float32)
    dR = np.empty((b, n_relations), np.float32)
    rc = _load().ora_follow_backward_residual(n_entities, n_relations, len(subj), _ptr(subj),
                                              _ptr(rel), _ptr(obj), _ptr(weight), b, _ptr(X),
                                              _ptr(R), _ptr(dY), gamma, _ptr(dX), _ptr(dR),
                                              nthreads)
    _check(rc, "follow_backward_residual")
    return dX, dR
