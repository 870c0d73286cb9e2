"""bench.py's own arithmetic and bookkeeping, on the CPU: the byte models of
the roofline entry (against counts done by hand on a small KB), the mapping
from batch width to the stream-kernel instance whose counters are looked up,
the fingerprint gate on committed traffic figures, and the one-GPU guard."""
import importlib.util
import json
import os
import subprocess
import sys
import types

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def small_kb():
    # 5 triples over 6 entities and 3 relations: subjects {0, 1, 4}, objects
    # {2, 3}; entity 5 appears nowhere.
    subj = np.array([0, 0, 1, 4, 4], np.int32)
    rel = np.array([0, 1, 1, 2, 2], np.int32)
    obj = np.array([2, 3, 3, 2, 2], np.int32)
    return types.SimpleNamespace(n_triples=5, n_entities=6, n_relations=3, subj=subj, rel=rel,
                                 obj=obj)


def test_byte_models_by_hand(bench):
    kb, b = small_kb(), 4
    row = 4 * b  # bytes of one b-wide float row
    ids = 8 * 5
    # forward: A = X rows of subjects, output rows = objects with triples
    g, c, o = bench.pass_bytes(kb, b, "fwd_stream")
    assert g == ids + 4 * 7 + 5 * row + 3 * row + 2 * row          # every triple's A row
    assert c == ids + 4 * 7 + 3 * row + 3 * row + 2 * row          # 3 distinct subjects
    assert o == ids + 4 * 7 + 6 * row + 3 * row + 2 * row          # all of X
    # dX: A = dY rows of objects, output rows = subjects with triples
    g, c, o = bench.pass_bytes(kb, b, "dx_stream")
    assert (g, c, o) == (ids + 28 + 5 * row + 3 * row + 3 * row,
                         ids + 28 + 2 * row + 3 * row + 3 * row,
                         ids + 28 + 6 * row + 3 * row + 3 * row)
    # dR: two gathered rows per triple; R-sized output
    g, c, o = bench.pass_bytes(kb, b, "dr_stream")
    assert (g, c, o) == (ids + 4 * 4 + 10 * row + 3 * row,
                         ids + 4 * 4 + (3 + 2) * row + 3 * row,
                         ids + 4 * 4 + 12 * row + 3 * row)
    # whole passes count the rows the zero fill writes too
    assert bench.pass_bytes(kb, b, "fwd_stream", whole_pass=True)[1] == \
        ids + 28 + 3 * row + 3 * row + 6 * row


def test_kernel_symbols_exist_in_the_build(bench):
    fp = os.path.join(ROOT, "paper_2002_06115_amd", "_lib", "kernels.fingerprint")
    if not os.path.exists(fp):
        pytest.skip("run __graft_entry__.build() first")
    digests = json.load(open(fp))
    for b in (1, 4, 5, 32, 128, 256, 300):
        for weighted in (False, True):
            for residual in (False, True):
                for plain, lds in ((False, False), (False, True), (True, False)):
                    sym = bench.stream_kernel_symbol(b, weighted, residual, plain, lds)
                    assert sym in digests, (b, weighted, residual, plain, lds, sym)


def test_committed_traffic_is_gated_by_the_fingerprint(bench, tmp_path, monkeypatch):
    sym = bench.stream_kernel_symbol(32)
    (tmp_path / "paper_2002_06115_amd" / "_lib").mkdir(parents=True)
    (tmp_path / "profiles").mkdir()
    prof = {"workload": "large", "batch": 32, "symbol": sym, "kernel_sha": "abc",
            "per_launch": {"dr_stream": {"bytes": 123.0}}}
    (tmp_path / "profiles" / "p.json").write_text(json.dumps(prof))
    fp = tmp_path / "paper_2002_06115_amd" / "_lib" / "kernels.fingerprint"
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    fp.write_text(json.dumps({sym: "abc"}))
    assert bench.measured_traffic("large", 32, "dr_stream", sym) == 123.0
    assert bench.measured_traffic("large", 32, "fwd_stream", sym) is None
    assert bench.measured_traffic("train", 32, "dr_stream", sym) is None
    fp.write_text(json.dumps({sym: "changed"}))  # the kernel was rebuilt differently
    assert bench.measured_traffic("large", 32, "dr_stream", sym) is None
    fp.unlink()
    assert bench.measured_traffic("large", 32, "dr_stream", sym) is None


def test_committed_profiles_match_the_built_kernels(bench):
    """The traffic figures in profiles/ were taken on the stream kernels built
    now (otherwise bench.py reports traffic as null)."""
    fp = os.path.join(ROOT, "paper_2002_06115_amd", "_lib", "kernels.fingerprint")
    if not os.path.exists(fp):
        pytest.skip("run __graft_entry__.build() first")
    import kbgen
    for workload in ("large", "train"):
        w = kbgen.WORKLOADS[workload]
        b = w.batch
        for phase, rows in (("fwd_stream", w.n_relations), ("dx_stream", w.n_relations),
                            ("dr_stream", w.n_entities)):
            lpt, lds = bench.stream_launch(b, rows)
            sym = bench.stream_kernel_symbol(b, lds=lds, lpt=lpt)
            assert bench.measured_traffic(workload, b, phase, sym) is not None, (workload, phase)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0 and "one GPU" in r.stderr


def test_stream_launch_mirrors_the_library_rule(bench):
    """bench.stream_launch: (lanes per group, B in LDS) for a pass whose B
    table has b_rows rows, as the library's launcher chooses it for the hard
    KB: the default layout when B's slice fits 80 KB, 32-column slices when
    that makes it fit 160 KB, registers otherwise."""
    assert bench.stream_launch(32, 600) == (8, True)        # 76.8 KB
    assert bench.stream_launch(32, 1280) == (8, True)       # 160 KB, one workgroup per CU
    assert bench.stream_launch(32, 1281) == (8, False)
    assert bench.stream_launch(128, 160) == (32, True)      # 80 KB at 128 columns
    assert bench.stream_launch(128, 161) == (8, True)       # cut into 32-column slices
    assert bench.stream_launch(256, 1000) == (8, True)      # 128 KB per 32-column slice
    assert bench.stream_launch(256, 10_000_000) == (32, False)
    assert bench.stream_launch(256, 1000, hard=False) == (32, False)
    assert bench.stream_kernel_symbol(256, lds=True, lpt=8) == \
        "_ZN3kbf12_GLOBAL__N_113stream_kernelILi4ELi8ELb1ELb0ELb0ELb1EEEvNS_10StreamArgsE"


def test_overlap_backward_rule(bench, monkeypatch):
    """bench's mirror of the library's rule for the concurrent backward."""
    monkeypatch.delenv("KBFOLLOW_OVERLAP_BACKWARD", raising=False)
    assert not bench.overlap_backward((1 << 20) - 1, 32)
    assert bench.overlap_backward(1 << 20, 32)
    assert not bench.overlap_backward(1 << 20, 64)
    monkeypatch.setenv("KBFOLLOW_OVERLAP_BACKWARD", "0")
    assert not bench.overlap_backward(50_000_000, 32)
    monkeypatch.setenv("KBFOLLOW_OVERLAP_BACKWARD", "1")
    assert bench.overlap_backward(5000, 256)
