"""Host side of the transfer engine's C ABI (no GPU): record sizes, argument
checks that reject bad index lists before any launch, and the C++ prefetch
plan against the oracle's, bit for bit."""
import ctypes
import os

import numpy as np
import pytest

import oracle.foremoe_transfer as X

FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first


@pytest.fixture(scope="module")
def lib():
    import paper_2606_11867_amd as fm
    if not os.path.exists(fm.LIB_PATH):
        from paper_2606_11867_amd import build
        build.build()
    return fm.load()


def test_record_bytes_match_the_oracle(lib):
    for d, F in ((2048, 768), (4096, 14336), (8, 4)):
        for what in (1, 2, 3):
            assert lib.foremoe_xfer_record_bytes(d, F, 1, what) == X.record_bytes(d, F, 2, what)
            assert lib.foremoe_xfer_record_bytes(d, F, 0, what) == X.record_bytes(d, F, 4, what)
    assert lib.foremoe_xfer_record_bytes(8, 4, 1, 0) == 0
    assert lib.foremoe_xfer_record_bytes(0, 4, 1, 3) == 0


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def test_copy_out_rejects_bad_lists(lib):
    w = _i32([0, 5])
    g = _i32([0, 1])
    rb = X.record_bytes(8, 4, 2, 3)
    # widx 5 outside W = 4
    assert lib.foremoe_copy_out(FAKE, FAKE, 1, 4, FAKE, FAKE, 2, 8, 4, 2, w.ctypes.data, g.ctypes.data, 3, FAKE,
                                2 * rb, None) == -1
    assert b"widx[1]" in lib.foremoe_last_error()
    # buffer too small
    w = _i32([0, 1])
    assert lib.foremoe_copy_out(FAKE, FAKE, 1, 4, FAKE, FAKE, 2, 8, 4, 2, w.ctypes.data, g.ctypes.data, 3, FAKE,
                                2 * rb - 1, None) == -1
    # too many records, bad part set, d*F not a multiple of 8
    assert lib.foremoe_copy_out(FAKE, FAKE, 1, 4, FAKE, FAKE, 2, 8, 4, 65, w.ctypes.data, g.ctypes.data, 3, FAKE,
                                1 << 30, None) == -1
    assert lib.foremoe_copy_out(FAKE, FAKE, 1, 4, FAKE, FAKE, 2, 8, 4, 2, w.ctypes.data, g.ctypes.data, 4, FAKE,
                                1 << 30, None) == -1
    assert lib.foremoe_copy_out(FAKE, FAKE, 1, 4, FAKE, FAKE, 2, 3, 3, 2, w.ctypes.data, g.ctypes.data, 3, FAKE,
                                1 << 30, None) == -2
    # nothing to do
    assert lib.foremoe_copy_out(None, None, 1, 4, None, None, 2, 8, 4, 0, None, None, 3, None, 0, None) == 0


def test_copy_in_rejects_bad_lists(lib):
    rb = X.record_bytes(8, 4, 2, 3)
    w, g, m = _i32([1, 1]), _i32([0, 1]), _i32([0, 1])
    # two records into one weight slot
    assert lib.foremoe_copy_in(FAKE, 2 * rb, 2, w.ctypes.data, g.ctypes.data, m.ctypes.data, 3, FAKE, FAKE, 1, 4,
                               FAKE, FAKE, 2, 8, 4, None) == -1
    assert b"weight slot 1" in lib.foremoe_last_error()
    w = _i32([0, 1])
    bad_mode = _i32([0, 7])
    assert lib.foremoe_copy_in(FAKE, 2 * rb, 2, w.ctypes.data, g.ctypes.data, bad_mode.ctypes.data, 3, FAKE, FAKE,
                               1, 4, FAKE, FAKE, 2, 8, 4, None) == -1
    g_bad = _i32([0, 2])
    assert lib.foremoe_copy_in(FAKE, 2 * rb, 2, w.ctypes.data, g_bad.ctypes.data, m.ctypes.data, 3, FAKE, FAKE, 1,
                               4, FAKE, FAKE, 2, 8, 4, None) == -1


def test_prefetch_rejects_bad_lists(lib):
    e, w = _i32([0, 9]), _i32([0, 1])
    assert lib.foremoe_prefetch_experts(FAKE, FAKE, 8, 1, 8, 4, 2, e.ctypes.data, w.ctypes.data, FAKE, FAKE, 4,
                                        None) == -1  # expert 9 outside E = 8
    e, w = _i32([0, 1]), _i32([2, 2])
    assert lib.foremoe_prefetch_experts(FAKE, FAKE, 8, 1, 8, 4, 2, e.ctypes.data, w.ctypes.data, FAKE, FAKE, 4,
                                        None) == -1  # one slot twice


def test_plan_prefetch_matches_the_oracle():
    from paper_2606_11867_amd import api
    slot_of, fe, fw = api.plan_prefetch([3, 7, -1, 5], [5, 2, 3, 9])
    assert slot_of.tolist() == [3, 1, 0, 2] and list(zip(fe.tolist(), fw.tolist())) == [(2, 1), (9, 2)]
    rng = np.random.default_rng(0)
    for _ in range(300):
        W, E = int(rng.integers(1, 24)), 40
        resident = [int(e) if rng.random() < 0.8 else -1 for e in rng.integers(0, E, size=W)]
        needed = [int(e) for e in rng.permutation(E)[:int(rng.integers(0, W + 1))]]
        so_o, f_o = X.plan_prefetch(resident, needed)
        so_g, fe, fw = api.plan_prefetch(resident, needed)
        assert so_g.tolist() == so_o
        assert list(zip(fe.tolist(), fw.tolist())) == f_o
    from paper_2606_11867_amd._lib import ForeMoEError
    with pytest.raises(ForeMoEError):
        api.plan_prefetch([0, 1], [2, 3, 4])
    with pytest.raises(ForeMoEError):
        api.plan_prefetch([0, 1], [2, 2])
