"""Host-side checks of the C-ABI library (no GPU needed).

The shared library must load, export every entry point include/kbfollow.h
declares, validate arguments before touching the device, and build the three
sorted layouts of the reified KB (Sec. 2.3) correctly.
"""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kbfollow.h")


@pytest.fixture(scope="module")
def kbf():
    import paper_2002_06115_amd as kbf
    return kbf


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kb_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("kb_create", "kb_destroy", "kb_workspace_size", "kb_follow", "kb_follow_backward",
              "kb_status_str", "kb_last_error", "kb_layout_host", "kb_get_info"):
        assert n in names


def test_library_exports_every_declared_symbol(kbf):
    lib = ctypes.CDLL(kbf.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_normal_build_has_no_bounds_checks(kbf):
    count = ctypes.c_uint64(7)
    assert kbf._lib.kb_checked_violations(ctypes.byref(count), 0) == kbf.KB_ENOTSUP
    assert count.value == 0
    with pytest.raises(kbf.KBError):
        kbf.checked_violations()


def test_checked_build_exports_every_declared_symbol():
    from paper_2002_06115_amd import build as kbuild
    lib = ctypes.CDLL(kbuild.CHECKED_LIB)
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings(kbf):
    lib = kbf._lib
    assert lib.kb_status_str(0) == b"ok"
    assert lib.kb_status_str(2) == b"id out of range"
    assert lib.kb_workspace_size(None, 4) == 0


def _create(kbf, n_e, n_r, s, r, o):
    h = ctypes.c_void_p()
    arr = [np.ascontiguousarray(a, np.int32) for a in (s, r, o)]
    st = kbf._lib.kb_create(n_e, n_r, len(arr[0]), *(a.ctypes.data_as(ctypes.c_void_p) for a in arr),
                            None, None, ctypes.byref(h))
    return st, h


@pytest.mark.parametrize("case,status", [
    (dict(s=[0, 5], r=[0, 0], o=[1, 1]), 2),       # subject id == N_E
    (dict(s=[0, 1], r=[0, 3], o=[1, 1]), 2),       # relation id == N_R
    (dict(s=[0, 1], r=[0, 0], o=[-1, 1]), 2),      # negative object id
])
def test_create_rejects_bad_ids_before_device_work(kbf, case, status):
    st, h = _create(kbf, 5, 3, case["s"], case["r"], case["o"])
    assert st == status and not h.value
    assert b"out of range" in kbf._lib.kb_last_error()


def test_create_rejects_bad_sizes(kbf):
    h = ctypes.c_void_p()
    assert kbf._lib.kb_create(-1, 1, 0, None, None, None, None, None, ctypes.byref(h)) == 1
    assert kbf._lib.kb_create(4, 1, 3, None, None, None, None, None, ctypes.byref(h)) == 1
    assert kbf._lib.kb_create(4, 1, 1 << 31, None, None, None, None, None, ctypes.byref(h)) == 1
    assert kbf._lib.kb_create(4, 1, 0, None, None, None, None, None, None) == 1


def test_layout_host_sorted_and_consistent(kbf):
    g = np.random.default_rng(5)
    n_e, n_r, n_t = 300, 7, 4000
    s = g.integers(0, n_e, n_t).astype(np.int32)
    r = g.integers(0, n_r, n_t).astype(np.int32)
    o = g.integers(0, n_e, n_t).astype(np.int32)
    specs = {0: (o, r, s, s, r), 1: (s, r, o, o, r), 2: (r, s, o, o, s)}
    for which, (k1, k2, k3, ca_src, cb_src) in specs.items():
        off, ca, cb, perm = kbf.layout_host(s, r, o, n_e, n_r, which)
        assert sorted(perm.tolist()) == list(range(n_t))
        assert np.array_equal(ca, ca_src[perm]) and np.array_equal(cb, cb_src[perm])
        want = np.lexsort((np.arange(n_t), k3, k2, k1))   # stable by (k1, k2, k3)
        assert np.array_equal(perm, want)
        rows = n_r if which == 2 else n_e
        assert np.array_equal(off, np.concatenate([[0], np.cumsum(np.bincount(k1, minlength=rows))]))


def test_layout_host_empty_and_duplicates(kbf):
    off, ca, cb, perm = kbf.layout_host(np.zeros(0), np.zeros(0), np.zeros(0), 4, 2, 0)
    assert np.array_equal(off, np.zeros(5)) and len(perm) == 0
    s = np.array([0, 0, 0], np.int32)
    off, ca, cb, perm = kbf.layout_host(s, s, s, 1, 1, 1)
    assert np.array_equal(off, [0, 3]) and np.array_equal(perm, [0, 1, 2])


def test_product_path_has_no_cpu_fallback():
    # The binding must not reach for the oracle or any CPU implementation.
    src = open(os.path.join(ROOT, "paper_2002_06115_amd", "__init__.py")).read()
    assert "oracle" not in src.replace("oracle.", "")  # no import of the oracle package
    assert "import oracle" not in src and "from oracle" not in src


@pytest.mark.parametrize("threads", ["1", "2", "5", "16"])
def test_layout_sort_same_for_any_thread_count(kbf, threads, monkeypatch):
    """The radix sorts split each pass over host threads (contiguous blocks,
    per-thread digit buckets): the order must be the stable (k1, k2, k3) order
    whatever the thread count.  300 k triples: several blocks per pass."""
    monkeypatch.setenv("KBFOLLOW_HOST_THREADS", threads)
    g = np.random.default_rng(17)
    n_e, n_r, n_t = 50_000, 40, 300_000
    s = np.minimum(g.zipf(1.3, n_t) - 1, n_e - 1).astype(np.int32)
    r = g.integers(0, n_r, n_t).astype(np.int32)
    o = g.integers(0, n_e, n_t).astype(np.int32)
    specs = {0: (o, r, s), 1: (s, r, o), 2: (r, s, o)}
    for which, (k1, k2, k3) in specs.items():
        off, ca, cb, perm = kbf.layout_host(s, r, o, n_e, n_r, which)
        assert np.array_equal(perm, np.lexsort((np.arange(n_t), k3, k2, k1))), which


def test_host_ids_refuse_ids_that_do_not_fit_int32(kbf):
    """An int64 id of 2^32 + 5 must not wrap to 5 (a different, in-range KB)."""
    with pytest.raises(ValueError):
        kbf._host_ids(np.array([0, (1 << 32) + 5], np.int64), 2)
    with pytest.raises(ValueError):
        kbf._host_ids(np.array([-(1 << 31) - 1], np.int64), 1)
    with pytest.raises(TypeError):
        kbf._host_ids(np.array([1.0, 2.0]), 2)
    ids = kbf._host_ids(np.array([3, 1 << 29], np.int64), 2)
    assert ids.dtype == np.int32 and list(ids) == [3, 1 << 29]
    assert kbf._host_ids([], 0).dtype == np.int32
    # Negative ids that fit int32 reach kb_create's own range check (KB_ERANGE).
    assert list(kbf._host_ids(np.array([-5], np.int64), 1)) == [-5]


def test_noalloc_scratch_limit_matches_the_library():
    """The header's KB_NOALLOC_SCRATCH_BYTES is the scratch size the library refuses beyond."""
    text = open(HEADER).read()
    m = re.search(r"#define KB_NOALLOC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", text)
    assert m, "KB_NOALLOC_SCRATCH_BYTES not found"
    src = open(os.path.join(ROOT, "paper_2002_06115_amd", "csrc", "kernels.h")).read()
    m2 = re.search(r"kStaticScratchBytes = size_t\((\d+)\) << (\d+);", src)
    assert m2 and (int(m.group(1)) << int(m.group(2))) == (int(m2.group(1)) << int(m2.group(2)))
