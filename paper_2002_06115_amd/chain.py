"""ctypes binding of the multi-hop chain glue (include/kbchain.h, libkbchain.so).

The column-wise steps between the hops of the multi-hop model of Sec. 3.2:
relation sets r^t = softmax(rho^t), per-example L1 normalisation of each hop's
entity weights, and the softmax cross-entropy of the last hop -- each with its
backward.  Every array is a contiguous float32 [n][b] CUDA tensor (one column
per example), as for the follow operation; reductions run in double on the
GPU.  Argument marshalling only: every step runs in the library's kernels.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("KBCHAIN_LIB", os.path.join(_HERE, "_lib", "libkbchain.so"))

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built: run paper_2002_06115_amd.build.build_chain() "
                      "(or __graft_entry__.build()) first")
_lib = ctypes.CDLL(LIB_PATH)
_P, _I64, _I32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
_lib.kbc_softmax.argtypes = [_I64, _I32, _P, _P, _P]
_lib.kbc_softmax_backward.argtypes = [_I64, _I32, _P, _P, _P, _P]
_lib.kbc_l1_normalize.argtypes = [_I64, _I32, _P, _P, _P, _P]
_lib.kbc_l1_normalize_backward.argtypes = [_I64, _I32, _P, _P, _P, _P, _P]
_lib.kbc_softmax_xent.argtypes = [_I64, _I32, _P, _P, _P, _P, _P, _P]
for _f in (_lib.kbc_softmax, _lib.kbc_softmax_backward, _lib.kbc_l1_normalize,
           _lib.kbc_l1_normalize_backward, _lib.kbc_softmax_xent):
    _f.restype = ctypes.c_int


def _mat(t, name, shape=None):
    import torch
    if not isinstance(t, torch.Tensor) or t.dtype != torch.float32 or not t.is_cuda:
        raise TypeError(f"{name} must be a float32 CUDA tensor")
    if t.dim() != 2 or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous [n][b] tensor")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}")
    return t


def _stream(t):
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _ok(status, what):
    if status != 0:
        raise RuntimeError(f"{what} failed with status {status}")


def softmax(z):
    """Column-wise softmax over the n rows: [n][b] -> [n][b]."""
    import torch
    z = _mat(z, "z")
    p = torch.empty_like(z)
    _ok(_lib.kbc_softmax(z.shape[0], z.shape[1], z.data_ptr(), p.data_ptr(), _stream(z)),
        "kbc_softmax")
    return p


def softmax_backward(p, dp):
    """dz = p * (dp - <dp, p>) per column, for p = softmax(z)."""
    import torch
    p = _mat(p, "p")
    dp = _mat(dp, "dp", p.shape)
    dz = torch.empty_like(p)
    _ok(_lib.kbc_softmax_backward(p.shape[0], p.shape[1], p.data_ptr(), dp.data_ptr(),
                                  dz.data_ptr(), _stream(p)), "kbc_softmax_backward")
    return dz


def l1_normalize(u):
    """(x, sums): x = u / sums with sums[beta] = sum of column beta (float64 [b])."""
    import torch
    u = _mat(u, "u")
    x = torch.empty_like(u)
    sums = torch.empty(u.shape[1], dtype=torch.float64, device=u.device)
    _ok(_lib.kbc_l1_normalize(u.shape[0], u.shape[1], u.data_ptr(), x.data_ptr(),
                              sums.data_ptr(), _stream(u)), "kbc_l1_normalize")
    return x, sums


def l1_normalize_backward(x, sums, dx):
    """du = (dx - <dx, x>) / sums per column."""
    import torch
    x = _mat(x, "x")
    dx = _mat(dx, "dx", x.shape)
    if sums.dtype != torch.float64 or sums.numel() != x.shape[1] or not sums.is_contiguous():
        raise ValueError("sums must be a contiguous float64 tensor of b elements")
    du = torch.empty_like(x)
    _ok(_lib.kbc_l1_normalize_backward(x.shape[0], x.shape[1], x.data_ptr(), sums.data_ptr(),
                                       dx.data_ptr(), du.data_ptr(), _stream(x)),
        "kbc_l1_normalize_backward")
    return du


def softmax_xent(z, t):
    """(loss, col_loss, dz): softmax cross-entropy of logits z against targets
    t, averaged over the b columns (loss: float64 0-d tensor, col_loss:
    float64 [b]), and dz = d loss / d z."""
    import torch
    z = _mat(z, "z")
    t = _mat(t, "t", z.shape)
    col = torch.empty(z.shape[1], dtype=torch.float64, device=z.device)
    loss = torch.empty((), dtype=torch.float64, device=z.device)
    dz = torch.empty_like(z)
    _ok(_lib.kbc_softmax_xent(z.shape[0], z.shape[1], z.data_ptr(), t.data_ptr(), col.data_ptr(),
                              loss.data_ptr(), dz.data_ptr(), _stream(z)), "kbc_softmax_xent")
    return loss, col, dz
