"""Event timing of the passes (kb_profile_enable / kb_profile_select): every
phase records one bracket per launch group, a phase mask records only the
phases it names, and recording off records nothing."""
import ctypes

import pytest

import kbgen
from gpu_util import to_em

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def setup():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2002_06115_amd as kbf
    w = kbgen.METAQA.scaled(20_000, 150_000, batch=32, tag=5)
    kb = kbgen.make_kb(w)
    gkb = kbf.KB(kb.subj, kb.rel, kb.obj, w.n_entities, w.n_relations)
    X, R, dY = to_em(kbgen.make_x(w)), to_em(kbgen.make_r(w)), to_em(kbgen.make_dy(w))
    yield kbf, gkb, X, R, dY
    gkb.close()


def step(gkb, X, R, dY):
    import torch
    gkb.follow(X, R)
    gkb.follow_backward(X, R, dY)
    torch.cuda.synchronize()


def test_all_phases(setup):
    kbf, gkb, X, R, dY = setup
    gkb.profile(True)
    step(gkb, X, R, dY)
    ph = gkb.profile_read()
    gkb.profile(False)
    info = gkb.info()
    for i, p in enumerate(("fwd", "dx", "dr")):
        ms, n = ph[f"{p}_stream"]
        assert n == 1 and ms > 0, p
        # one bracket around the tail launch, one around the further combine levels
        assert ph[f"{p}_tail"][1] == 1 and ph[f"{p}_combine"][1] == 1, p
        if info["n_levels"][i] > 1:
            assert ph[f"{p}_combine"][0] > 0, p


def test_phase_mask_records_only_named_phases(setup):
    kbf, gkb, X, R, dY = setup
    gkb.profile(True, phases=["dr_stream", "fwd_tail"])
    step(gkb, X, R, dY)
    step(gkb, X, R, dY)
    ph = gkb.profile_read()
    gkb.profile(False)
    assert {p for p, (ms, n) in ph.items() if n} == {"dr_stream", "fwd_tail"}
    assert ph["dr_stream"][1] == 2 and ph["dr_stream"][0] > 0


def test_off_records_nothing_and_bits_past_the_phases_are_ignored(setup):
    kbf, gkb, X, R, dY = setup
    gkb.profile(False)
    step(gkb, X, R, dY)
    assert all(n == 0 for ms, n in gkb.profile_read().values())
    lib = ctypes.CDLL(kbf.LIB_PATH)
    lib.kb_profile_select.argtypes = [ctypes.c_void_p, ctypes.c_uint32]
    assert lib.kb_profile_select(gkb._handle, 0xFFFFFFFF) == 0
    step(gkb, X, R, dY)
    ph = gkb.profile_read()
    assert all(n == 1 for ms, n in ph.values())
    gkb.profile(False)
