"""Relation-set following on a reified knowledge base, for MI355X (gfx950).

A thin ctypes binding over ``libkbfollow.so`` (declared in
``include/kbfollow.h``): argument marshalling only, every step of the
computation runs in the library's HIP kernels.  PyTorch supplies device memory
and the current stream.

    kb = KB(subj, rel, obj, n_entities, n_relations)        # host int32 triples
    Y  = kb.follow(X, R)                                    # X [N_E][b], R [N_R][b]
    dX, dR = kb.follow_backward(X, R, dY)
    Y  = follow(kb, X, R)                                   # autograd-aware
    Y  = follow_residual(kb, X, R)                          # follow(X, R) + X (App. E)

Activations are entity-major and batch-contiguous float32 CUDA tensors:
``X[i, beta]`` is the weight of entity i in example beta (the transpose of the
paper's ``b x N_E`` minibatch, App. C).  The library never falls back to any
other implementation: if it is not built, importing this module raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("KBFOLLOW_LIB") or os.path.join(_PKG, "_lib", "libkbfollow.so")

KB_OK, KB_EINVAL, KB_ERANGE, KB_ENOMEM, KB_EHIP, KB_ENOTSUP = range(6)
PHASES = ("fwd_stream", "fwd_tail", "fwd_combine", "dx_stream", "dx_tail", "dx_combine",
          "dr_stream", "dr_tail", "dr_combine")


class KBError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{message} (status {status})")
        self.status = status


class KBInfo(ctypes.Structure):
    _fields_ = [("n_entities", ctypes.c_int64), ("n_relations", ctypes.c_int64),
                ("n_triples", ctypes.c_int64), ("weighted", ctypes.c_int32),
                ("chunk_len", ctypes.c_int32 * 3), ("n_chunks", ctypes.c_int64 * 3),
                ("n_split_rows", ctypes.c_int64 * 3), ("n_slots", ctypes.c_int64 * 3),
                ("n_levels", ctypes.c_int32 * 3), ("n_empty_rows", ctypes.c_int64 * 3),
                ("max_row_len", ctypes.c_int64 * 3), ("device_bytes", ctypes.c_int64)]

    def as_dict(self):
        d = {}
        for name, _ in self._fields_:
            v = getattr(self, name)
            d[name] = list(v) if hasattr(v, "__len__") else int(v)
        return d


def _load_library():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2002_06115_amd.build` "
                          "(or __graft_entry__.build()) first")
    lib = ctypes.CDLL(LIB_PATH)
    i64, i32, p, sz = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p, ctypes.c_size_t
    lib.kb_create.argtypes = [i64, i64, i64, p, p, p, p, p, ctypes.POINTER(p)]
    lib.kb_create.restype = ctypes.c_int
    lib.kb_destroy.argtypes = [p]
    lib.kb_destroy.restype = None
    lib.kb_workspace_size.argtypes = [p, i32]
    lib.kb_workspace_size.restype = sz
    lib.kb_follow.argtypes = [p, i32, p, p, p, p, sz, p]
    lib.kb_follow.restype = ctypes.c_int
    lib.kb_follow_backward.argtypes = [p, i32, p, p, p, p, p, p, sz, p]
    lib.kb_follow_backward.restype = ctypes.c_int
    lib.kb_follow_noalloc.argtypes = [p, i32, p, p, p, p]
    lib.kb_follow_noalloc.restype = ctypes.c_int
    f32 = ctypes.c_float
    lib.kb_follow_residual.argtypes = [p, i32, p, p, f32, p, p, sz, p]
    lib.kb_follow_residual.restype = ctypes.c_int
    lib.kb_follow_accumulate.argtypes = [p, i32, p, p, p, f32, p, p, sz, p]
    lib.kb_follow_accumulate.restype = ctypes.c_int
    lib.kb_follow_backward_residual.argtypes = [p, i32, p, p, p, f32, p, p, p, sz, p]
    lib.kb_follow_backward_residual.restype = ctypes.c_int
    lib.kb_status_str.argtypes = [ctypes.c_int]
    lib.kb_status_str.restype = ctypes.c_char_p
    lib.kb_last_error.argtypes = []
    lib.kb_last_error.restype = ctypes.c_char_p
    lib.kb_get_info.argtypes = [p, ctypes.POINTER(KBInfo)]
    lib.kb_get_info.restype = ctypes.c_int
    lib.kb_layout_host.argtypes = [i64, i64, i64, p, p, p, i32, p, p, p, p]
    lib.kb_layout_host.restype = ctypes.c_int
    lib.kb_profile_enable.argtypes = [p, i32]
    lib.kb_profile_enable.restype = ctypes.c_int
    lib.kb_profile_select.argtypes = [p, ctypes.c_uint32]
    lib.kb_profile_select.restype = ctypes.c_int
    lib.kb_profile_read.argtypes = [p, p, p]
    lib.kb_profile_read.restype = ctypes.c_int
    lib.kb_phase_kernel.argtypes = [p, i32, i32, i32, ctypes.c_char_p, sz]
    lib.kb_phase_kernel.restype = ctypes.c_int
    lib.kb_checked_violations.argtypes = [ctypes.POINTER(ctypes.c_uint64), i32]
    lib.kb_checked_violations.restype = ctypes.c_int
    return lib


_lib = _load_library()


def _check(status, what):
    if status != KB_OK:
        detail = _lib.kb_last_error().decode()
        raise KBError(status, f"{what}: {_lib.kb_status_str(status).decode()}: {detail}")


def _host_ids(a, n):
    """A contiguous int32 copy (or view) of an id array; ids that do not fit
    int32 are rejected here rather than wrapped into a different, in-range id."""
    a = np.asarray(a)
    if a.shape != (n,):
        raise ValueError("subj, rel and obj must be 1-D arrays of equal length")
    if a.size == 0:
        return np.empty(0, np.int32)
    if a.dtype != np.int32:
        if not np.issubdtype(a.dtype, np.integer):
            raise TypeError(f"ids must be integers, got {a.dtype}")
        if int(a.min()) < np.iinfo(np.int32).min or int(a.max()) > np.iinfo(np.int32).max:
            raise ValueError("ids must fit int32 (the library takes ids below 2^30)")
        a = a.astype(np.int32)
    return np.ascontiguousarray(a)


def _np_ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def checked_violations(reset=False):
    """Index violations a checked build (KBFOLLOW_CHECKED) has counted on the
    current device; raises KBError (KB_ENOTSUP) for a normal build."""
    count = ctypes.c_uint64()
    _check(_lib.kb_checked_violations(ctypes.byref(count), 1 if reset else 0),
           "kb_checked_violations")
    return int(count.value)


def layout_host(subj, rel, obj, n_entities, n_relations, which):
    """The sorted layout the library builds (host only): (offsets, col_a, col_b, perm)."""
    n_t = len(subj)
    subj, rel, obj = (_host_ids(a, n_t) for a in (subj, rel, obj))
    rows = n_relations if which == 2 else n_entities
    off = np.empty(rows + 1, np.int32)
    ca, cb, perm = (np.empty(n_t, np.int32) for _ in range(3))
    _check(_lib.kb_layout_host(n_entities, n_relations, n_t, _np_ptr(subj), _np_ptr(rel),
                               _np_ptr(obj), which, _np_ptr(off), _np_ptr(ca), _np_ptr(cb),
                               _np_ptr(perm)), "kb_layout_host")
    return off, ca, cb, perm


class KB:
    """A reified KB resident on one GPU (Sec. 2.3): N_T triples (subj, rel, obj)."""

    def __init__(self, subj, rel, obj, n_entities, n_relations, weight=None, device=None):
        import torch
        n_t = len(subj)
        subj, rel, obj = (_host_ids(a, n_t) for a in (subj, rel, obj))
        w = None if weight is None else np.ascontiguousarray(weight, dtype=np.float32)
        if w is not None and w.shape != (n_t,):
            raise ValueError("weight must have one entry per triple")
        self.device = torch.device("cuda", torch.cuda.current_device()) if device is None \
            else torch.device(device)
        self.n_entities, self.n_relations, self.n_triples = int(n_entities), int(n_relations), n_t
        self._ws = {}
        self._handle = ctypes.c_void_p()
        with torch.cuda.device(self.device):
            stream = torch.cuda.current_stream(self.device).cuda_stream
            _check(_lib.kb_create(self.n_entities, self.n_relations, n_t, _np_ptr(subj),
                                  _np_ptr(rel), _np_ptr(obj), _np_ptr(w), ctypes.c_void_p(stream),
                                  ctypes.byref(self._handle)), "kb_create")

    def close(self):
        if getattr(self, "_handle", None) and self._handle.value:
            import torch
            torch.cuda.synchronize(self.device)
            _lib.kb_destroy(self._handle)
            self._handle = ctypes.c_void_p()
            self._ws.clear()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- helpers -------------------------------------------------------------
    def info(self):
        inf = KBInfo()
        _check(_lib.kb_get_info(self._handle, ctypes.byref(inf)), "kb_get_info")
        return inf.as_dict()

    def workspace_size(self, b):
        return int(_lib.kb_workspace_size(self._handle, int(b)))

    def workspace(self, b, stream=None):
        """A cached device workspace for batch size b on `stream` (uint8 tensor
        or None).  Each stream gets its own, so calls on different streams can
        run at the same time (calls on one stream are ordered by it)."""
        import torch
        n = self.workspace_size(b)
        if n == 0:
            return None
        s = torch.cuda.current_stream(self.device) if stream is None else stream
        key = (b, s.cuda_stream)
        ws = self._ws.get(key)
        if ws is None or ws.numel() < n:
            with torch.cuda.stream(s):
                ws = torch.empty(n, dtype=torch.uint8, device=self.device)
            self._ws[key] = ws
        return ws

    def _act(self, t, rows, name):
        import torch
        if t is None:
            return None
        if not isinstance(t, torch.Tensor) or t.dtype != torch.float32 or t.device != self.device:
            raise TypeError(f"{name} must be a float32 tensor on {self.device}")
        if t.dim() != 2 or t.shape[0] != rows or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous [{rows}][b] tensor")
        return t

    @staticmethod
    def _ptr(t):
        return None if t is None else ctypes.c_void_p(t.data_ptr())

    # -- the operations --------------------------------------------------------
    def follow(self, X, R, out=None, stream=None, residual=None):
        """Y = follow(X, R) (Eq. 4) for X [N_E][b], R [N_R][b]; returns Y [N_E][b].

        With ``residual=gamma``: Y = follow(X, R) + gamma * X, the hop of the
        KB-completion chains (Sec. 3.2, App. E).
        """
        import torch
        X = self._act(X, self.n_entities, "X")
        R = self._act(R, self.n_relations, "R")
        b = X.shape[1]
        if R.shape[1] != b:
            raise ValueError("X and R must have the same batch size")
        Y = torch.empty_like(X) if out is None else self._act(out, self.n_entities, "out")
        s = torch.cuda.current_stream(self.device) if stream is None else stream
        ws = self.workspace(b, s)
        nws = 0 if ws is None else ws.numel()
        with torch.cuda.device(self.device):
            if residual is None:
                _check(_lib.kb_follow(self._handle, b, self._ptr(X), self._ptr(R), self._ptr(Y),
                                      self._ptr(ws), nws, ctypes.c_void_p(s.cuda_stream)),
                       "kb_follow")
            else:
                _check(_lib.kb_follow_residual(self._handle, b, self._ptr(X), self._ptr(R),
                                               float(residual), self._ptr(Y), self._ptr(ws), nws,
                                               ctypes.c_void_p(s.cuda_stream)),
                       "kb_follow_residual")
        return Y

    def follow_noalloc(self, X, R, out, stream=None):
        """follow(X, R) into the caller's ``out`` through kb_follow_noalloc:
        the split-row partials use the library's fixed per-GPU scratch, so
        neither this call nor the library allocates.  Calls that overlap on
        one GPU share that scratch and must not be issued."""
        X = self._act(X, self.n_entities, "X")
        R = self._act(R, self.n_relations, "R")
        Y = self._act(out, self.n_entities, "out")
        b = X.shape[1]
        if R.shape[1] != b or Y.shape[1] != b:
            raise ValueError("X, R and out must have the same batch size")
        import torch
        s = torch.cuda.current_stream(self.device) if stream is None else stream
        with torch.cuda.device(self.device):
            _check(_lib.kb_follow_noalloc(self._handle, b, self._ptr(X), self._ptr(R),
                                          self._ptr(Y), ctypes.c_void_p(s.cuda_stream)),
                   "kb_follow_noalloc")
        return Y

    def follow_accumulate(self, X, R, Z, gamma=1.0, out=None, stream=None):
        """Y = follow(X, R) + gamma * Z for Z [N_E][b]; ``out=Z`` adds the hop
        into Z in place.  The gradient with respect to Z is gamma * dY."""
        import torch
        X = self._act(X, self.n_entities, "X")
        R = self._act(R, self.n_relations, "R")
        Z = self._act(Z, self.n_entities, "Z")
        b = X.shape[1]
        if R.shape[1] != b or Z.shape[1] != b:
            raise ValueError("X, R and Z must have the same batch size")
        Y = torch.empty_like(X) if out is None else self._act(out, self.n_entities, "out")
        s = torch.cuda.current_stream(self.device) if stream is None else stream
        ws = self.workspace(b, s)
        nws = 0 if ws is None else ws.numel()
        with torch.cuda.device(self.device):
            _check(_lib.kb_follow_accumulate(self._handle, b, self._ptr(X), self._ptr(R),
                                             self._ptr(Z), float(gamma), self._ptr(Y),
                                             self._ptr(ws), nws, ctypes.c_void_p(s.cuda_stream)),
                   "kb_follow_accumulate")
        return Y

    def follow_backward(self, X, R, dY, want_dx=True, want_dr=True, dX=None, dR=None,
                        stream=None, residual=None):
        """(dX [N_E][b], dR [N_R][b]) for upstream gradient dY [N_E][b].

        With ``residual=gamma`` the gradients of follow(X, R) + gamma * X
        (dX gains gamma * dY).
        """
        import torch
        dY = self._act(dY, self.n_entities, "dY")
        b = dY.shape[1]
        X = self._act(X, self.n_entities, "X") if want_dr else None
        R = self._act(R, self.n_relations, "R") if want_dx else None
        if want_dx and dX is None:
            dX = torch.empty((self.n_entities, b), dtype=torch.float32, device=self.device)
        if want_dr and dR is None:
            dR = torch.empty((self.n_relations, b), dtype=torch.float32, device=self.device)
        dX = self._act(dX, self.n_entities, "dX") if want_dx else None
        dR = self._act(dR, self.n_relations, "dR") if want_dr else None
        s = torch.cuda.current_stream(self.device) if stream is None else stream
        ws = self.workspace(b, s)
        nws = 0 if ws is None else ws.numel()
        with torch.cuda.device(self.device):
            if residual is None:
                _check(_lib.kb_follow_backward(self._handle, b, self._ptr(X), self._ptr(R),
                                               self._ptr(dY), self._ptr(dX), self._ptr(dR),
                                               self._ptr(ws), nws, ctypes.c_void_p(s.cuda_stream)),
                       "kb_follow_backward")
            else:
                _check(_lib.kb_follow_backward_residual(
                    self._handle, b, self._ptr(X), self._ptr(R), self._ptr(dY), float(residual),
                    self._ptr(dX), self._ptr(dR), self._ptr(ws), nws,
                    ctypes.c_void_p(s.cuda_stream)), "kb_follow_backward_residual")
        return dX, dR

    # -- event timing -----------------------------------------------------------
    def profile(self, on=True, phases=None):
        """Record events around every phase's launches (on), none (off), or
        only the phases named in `phases` (names from PHASES)."""
        if phases is None:
            _check(_lib.kb_profile_enable(self._handle, 1 if on else 0), "kb_profile_enable")
            return
        mask = 0
        for p in phases:
            mask |= 1 << PHASES.index(p)
        _check(_lib.kb_profile_select(self._handle, mask if on else 0), "kb_profile_select")

    def phase_kernels(self, b, residual=False):
        """{phase: the kernel it launches at batch size b, as profilers print
        it ("" when the phase launches nothing)}."""
        out = {}
        buf = ctypes.create_string_buffer(256)
        for i, p in enumerate(PHASES):
            _check(_lib.kb_phase_kernel(self._handle, int(b), i, 1 if residual else 0, buf,
                                        len(buf)), "kb_phase_kernel")
            out[p] = buf.value.decode()
        return out

    def profile_read(self):
        """{phase: (total ms, launches)} since the last read."""
        ms = (ctypes.c_double * len(PHASES))()
        n = (ctypes.c_int64 * len(PHASES))()
        _check(_lib.kb_profile_read(self._handle, ctypes.cast(ms, ctypes.c_void_p),
                                    ctypes.cast(n, ctypes.c_void_p)), "kb_profile_read")
        return {p: (ms[i], n[i]) for i, p in enumerate(PHASES)}


def _make_functions():
    import torch

    class _Follow(torch.autograd.Function):
        @staticmethod
        def forward(ctx, X, R, kb, residual):
            ctx.kb = kb
            ctx.residual = residual
            ctx.save_for_backward(X, R)
            return kb.follow(X, R, residual=residual)

        @staticmethod
        def backward(ctx, dY):
            X, R = ctx.saved_tensors
            need_x, need_r = ctx.needs_input_grad[0], ctx.needs_input_grad[1]
            dX, dR = ctx.kb.follow_backward(X, R, dY.contiguous(), want_dx=need_x,
                                            want_dr=need_r, residual=ctx.residual)
            return dX, dR, None, None

    return _Follow


_FollowFn = None


def follow(kb: KB, X, R):
    """Differentiable follow(X, R) (Eq. 4) on entity-major tensors X [N_E][b], R [N_R][b]."""
    global _FollowFn
    if _FollowFn is None:
        _FollowFn = _make_functions()
    return _FollowFn.apply(X, R, kb, None)


def follow_residual(kb: KB, X, R, gamma: float = 1.0):
    """Differentiable residual hop follow(X, R) + gamma * X (Sec. 3.2, App. E)."""
    global _FollowFn
    if _FollowFn is None:
        _FollowFn = _make_functions()
    return _FollowFn.apply(X, R, kb, float(gamma))


__all__ = ["KB", "KBError", "follow", "follow_residual", "layout_host", "LIB_PATH", "PHASES"]
