"""bench.py's own arithmetic and bookkeeping, on the CPU: the byte models of
the roofline entry (against counts done by hand on a small KB), the mapping
from a kernel's profiler name to its symbol in the build, the fingerprint gate
on committed traffic figures, and the one-GPU guard."""
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
    m = bench.pass_bytes(kb, b, "fwd")
    assert m["gather"] == ids + 4 * 7 + 5 * row + 3 * row + 2 * row      # every triple's A row
    assert m["distinct"] == ids + 4 * 7 + 3 * row + 3 * row + 2 * row    # 3 distinct subjects
    assert m["array_once"] == ids + 4 * 7 + 6 * row + 3 * row + 2 * row  # all of X
    # dX: A = dY rows of objects, output rows = subjects with triples
    m = bench.pass_bytes(kb, b, "dx")
    assert (m["gather"], m["distinct"], m["array_once"]) == (
        ids + 28 + 5 * row + 3 * row + 3 * row, ids + 28 + 2 * row + 3 * row + 3 * row,
        ids + 28 + 6 * row + 3 * row + 3 * row)
    # dR: two gathered rows per triple; R-sized output
    m = bench.pass_bytes(kb, b, "dr")
    assert (m["gather"], m["distinct"], m["array_once"]) == (
        ids + 4 * 4 + 10 * row + 3 * row, ids + 4 * 4 + (3 + 2) * row + 3 * row,
        ids + 4 * 4 + 12 * row + 3 * row)
    # whole passes count the rows the zero fill writes too
    assert bench.pass_bytes(kb, b, "fwd", whole_pass=True)["distinct"] == \
        ids + 28 + 3 * row + 3 * row + 6 * row


def test_array_once_bytes_of_the_large_kb(bench):
    """The figures the roofline is judged by, for the 10 M-entity / 50 M-triple
    KB at b = 32: 2.365 GB per forward / dX stream-kernel launch (5.04 M
    output rows with triples), 3.00 GB per whole forward or dX pass, 2.96 GB
    for dR, 8.96 GB per step."""
    kb = types.SimpleNamespace(n_triples=50_000_000, n_entities=10_000_000, n_relations=600)
    bench._DISTINCT[id(kb)] = (5_035_558, 5_036_810)
    fwd = bench.pass_bytes(kb, 32, "fwd")["array_once"]
    assert abs(fwd - 2.3648e9) < 1e6
    step = sum(bench.pass_bytes(kb, 32, p, whole_pass=True)["array_once"]
               for p in ("fwd", "dx", "dr"))
    assert abs(step - 8.9602e9) < 1e6


def test_mangled_names_match_the_build(bench):
    """Profiler names map onto the build's kernel symbols (whose assembly
    digests gate the committed traffic figures)."""
    fp = os.path.join(ROOT, "paper_2002_06115_amd", "_lib", "kernels.fingerprint")
    if not os.path.exists(fp):
        pytest.skip("run __graft_entry__.build() first")
    digests = json.load(open(fp))
    for vec in (1, 4):
        for lpt in (1, 2, 4, 8, 16, 32):
            for flags in ("true, false, false, false", "true, false, false, true",
                          "true, true, false, false", "true, false, true, true",
                          "false, false, false, false", "false, true, true, false"):
                name = f"stream_kernel<{vec}, {lpt}, {flags}>"
                assert bench.mangled_name(name) in digests, name
            assert bench.mangled_name(f"tail_kernel<{vec}, {lpt}, true>") in digests
            assert bench.mangled_name(f"combine_kernel<{vec}, {lpt}>") in digests
    assert bench.mangled_name("stream_kernel<4, 8, true, false, false, true>") == \
        "_ZN3kbf12_GLOBAL__N_113stream_kernelILi4ELi8ELb1ELb0ELb0ELb1EEEvNS_10StreamArgsE"


def test_committed_traffic_is_gated_by_the_fingerprint(bench, tmp_path, monkeypatch):
    name = "stream_kernel<4, 8, true, false, false, false>"
    sym = bench.mangled_name(name)
    (tmp_path / "paper_2002_06115_amd" / "_lib").mkdir(parents=True)
    (tmp_path / "profiles").mkdir()
    prof = {"workload": "large", "batch": 32,
            "kernels": {"dr_stream": {"kernel": name, "kernel_sha": "abc"}},
            "per_launch": {"dr_stream": {"bytes": 123.0}}}
    (tmp_path / "profiles" / "p.json").write_text(json.dumps(prof))
    fp = tmp_path / "paper_2002_06115_amd" / "_lib" / "kernels.fingerprint"
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    fp.write_text(json.dumps({sym: "abc"}))
    assert bench.measured_traffic("large", 32, name, ["dr_stream"])[0] == 123.0
    assert bench.measured_traffic("large", 32, name, ["fwd_stream"])[0] is None
    assert bench.measured_traffic("large", 32, name, ["dr_stream", "fwd_stream"])[0] is None
    assert bench.measured_traffic("train", 32, name, ["dr_stream"])[0] is None
    fp.write_text(json.dumps({sym: "changed"}))  # the kernel was rebuilt differently
    assert bench.measured_traffic("large", 32, name, ["dr_stream"])[0] is None
    fp.unlink()
    assert bench.measured_traffic("large", 32, name, ["dr_stream"])[0] is None


def test_committed_profiles_match_the_built_kernels(bench):
    """Every kernel a committed profile gives counters for was taken on the
    device code built now (otherwise bench.py reports its traffic as null):
    re-take the counters after changing a kernel."""
    fp = os.path.join(ROOT, "paper_2002_06115_amd", "_lib", "kernels.fingerprint")
    if not os.path.exists(fp):
        pytest.skip("run __graft_entry__.build() first")
    digests = json.load(open(fp))
    import glob
    found = 0
    for path in glob.glob(os.path.join(ROOT, "profiles", "*.json")):
        prof = json.load(open(path))
        for phase, k in prof.get("kernels", {}).items():
            assert digests.get(bench.mangled_name(k["kernel"])) == k["kernel_sha"], \
                (os.path.basename(path), phase, k["kernel"])
            found += 1
    assert found > 0


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0 and "one GPU" in r.stderr


def test_overlap_backward_rule(bench, monkeypatch):
    """bench's mirror of the library's rule for the concurrent backward."""
    monkeypatch.delenv("KBFOLLOW_OVERLAP_BACKWARD", raising=False)
    assert not bench._overlap((1 << 20) - 1, 32)
    assert bench._overlap(1 << 20, 32)
    assert not bench._overlap(1 << 20, 64)
    monkeypatch.setenv("KBFOLLOW_OVERLAP_BACKWARD", "0")
    assert not bench._overlap(50_000_000, 32)
    monkeypatch.setenv("KBFOLLOW_OVERLAP_BACKWARD", "1")
    assert bench._overlap(5000, 256)


def test_timed_phases_leave_concurrent_dx_launches_alone(bench):
    """With the concurrent backward, a kernel that runs both the forward and
    dX is timed on its forward launches; dR alone, or any kernel when the
    passes run one after another, is timed on every launch."""
    both = ["fwd_stream", "dx_stream"]
    assert bench.timed_phases(both, True) == ["fwd_stream"]
    assert bench.timed_phases(both, False) == both
    assert bench.timed_phases(["dr_stream"], True) == ["dr_stream"]
    assert bench.timed_phases(["dx_stream"], True) == ["dx_stream"]
    assert bench.timed_phases(["fwd_stream", "dx_stream", "dr_stream"], True) == \
        ["fwd_stream", "dr_stream"]


def test_dominant_kernel_near_tie_prefers_a_kernel_with_launches_of_its_own(bench):
    """Shares within 5 %: with the concurrent backward the kernel whose
    launches all overlap another pass gives way; otherwise the larger share
    wins, and a clear winner keeps its place."""
    kernels = {"fwd_stream": "K1", "dx_stream": "K1", "dr_stream": "K2",
               "fwd_tail": "T", "dx_tail": "T", "dr_tail": "T"}
    phases = {"fwd_stream": (0.72, 1), "dx_stream": (0.82, 1), "dr_stream": (1.56, 1),
              "fwd_tail": (0.15, 1), "dx_tail": (0.69, 1), "dr_tail": (0.02, 1)}
    assert bench.dominant_kernel(kernels, phases, concurrent=True)[0] == "K1"
    assert bench.dominant_kernel(kernels, phases, concurrent=False)[0] == "K2"
    phases["dr_stream"] = (1.80, 1)
    assert bench.dominant_kernel(kernels, phases, concurrent=True)[0] == "K2"
