"""Helpers shared by the GPU parity tests: uploads, transposes and the tolerance check.

The oracle works in the paper's batch-major orientation [b][N]; the library in
entity-major [N][b].  Inputs are generated once (kbgen), handed to the oracle
as they are and to the GPU transposed.
"""
import numpy as np

RTOL, ATOL = 1e-5, 1e-7


def to_em(t_bm):
    """[b][N] numpy -> contiguous [N][b] float32 CUDA tensor."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(t_bm, np.float32)).cuda().t().contiguous()


def from_em(t_em):
    """[N][b] CUDA tensor -> [b][N] numpy."""
    return t_em.t().contiguous().cpu().numpy()


def tol_ratio(got, want):
    """max over elements of |got - want| / (ATOL + RTOL |want|); <= 1 passes."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    if got.size == 0:
        return 0.0
    return float((np.abs(got - want) / (ATOL + RTOL * np.abs(want))).max())


def assert_close(got, want, what=""):
    assert got.shape == want.shape, (what, got.shape, want.shape)
    assert np.all(np.isfinite(got)), what
    r = tol_ratio(got, want)
    assert r <= 1.0, f"{what}: max |gpu-oracle|/(atol+rtol|oracle|) = {r:.3g}"
    return r


def assert_bitexact(got, want, what=""):
    assert got.shape == want.shape, (what, got.shape, want.shape)
    bad = np.nonzero(got != want)
    assert bad[0].size == 0, f"{what}: {bad[0].size} elements differ, first at {tuple(x[0] for x in bad)}"
