"""Host-side checks of the C ABI: the library loads, exports every function
declared in include/foremoe.h, and rejects bad arguments before touching the
GPU (these calls return from host validation; no kernel is launched)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "foremoe.h")


@pytest.fixture(scope="module")
def lib():
    import paper_2606_11867_amd as fm
    if not os.path.exists(fm.LIB_PATH):
        from paper_2606_11867_amd import build
        build.build()
    return fm.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(foremoe_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_five_steps():
    names = declared_functions()
    for n in ["foremoe_histogram", "foremoe_assign_replicas", "foremoe_permute", "foremoe_grouped_ffn_fwd",
              "foremoe_grouped_ffn_dgrad", "foremoe_grouped_ffn_wgrad", "foremoe_combine",
              "foremoe_combine_bwd", "foremoe_permute_bwd"]:
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    from paper_2606_11867_amd import _lib
    for name in declared_functions():
        assert hasattr(lib, name), name
        assert name in _lib.SIGNATURES, f"{name} missing from the binding"


def test_version_and_status_strings(lib):
    assert b"gfx950" in lib.foremoe_version()
    assert lib.foremoe_status_string(0) == b"ok"
    assert lib.foremoe_status_string(-1) == b"invalid argument"
    assert lib.foremoe_status_string(-2) == b"unsupported shape or dtype"


def test_timed_row_gemms_check_like_the_plain_calls(lib):
    # the timed forms validate their arguments like the plain calls, before
    # any launch or event record; the ABI keeps no launch state
    assert not hasattr(lib, "foremoe_set_launch_events")
    ev = (None, None)
    assert lib.foremoe_ffn_gate_up_fwd_timed(FAKE, 1, 96, 256, 4, FAKE, FAKE, 3, FAKE, 64, FAKE, None, None, 0,
                                             None, *ev) == -2
    assert lib.foremoe_ffn_down_fwd_timed(FAKE, 7, 128, 256, 4, FAKE, FAKE, 3, FAKE, 64, FAKE, None, 0,
                                          None, *ev) == -1
    assert lib.foremoe_ffn_down_dgrad_timed(FAKE, FAKE, 1, 128, 200, 4, FAKE, FAKE, 3, FAKE, 64, FAKE, None, 0,
                                            None, *ev) == -2
    assert lib.foremoe_ffn_gate_up_dgrad_timed(FAKE, 1, 128, 256, 4, FAKE, FAKE, 3, FAKE, 64, FAKE, FAKE, 16,
                                               None, *ev) == -1  # workspace too small


def test_workspace_size(lib):
    small = lib.foremoe_workspace_size(256, 2, 8)
    assert small > 0 and small % 256 == 0
    big = lib.foremoe_workspace_size(32768, 8, 256)
    assert big > small
    # status words, the replica->slot table, the virtual-slot offsets
    # (1025 ints rounded to 256 bytes), then [blocks][E+1] partial counts
    # (one block per 512 pairs), then a uint16 in-block rank per pair
    fixed = 256 + 4 * 1024 * 16 + 4352
    need = fixed + 512 * 257 * 4 + 2 * 32768 * 8
    assert big >= need
    assert big - need < 512
    assert lib.foremoe_workspace_size(-1, 2, 8) == 0
    assert lib.foremoe_workspace_size(10, 0, 8) == 0
    assert lib.foremoe_workspace_size(10, 2, 2000) == 0


FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first


def test_histogram_rejects_bad_args(lib):
    assert lib.foremoe_histogram(None, 10, 2, 8, FAKE, FAKE, 1 << 20, None) == -1
    assert lib.foremoe_histogram(FAKE, 10, 0, 8, FAKE, FAKE, 1 << 20, None) == -1
    assert lib.foremoe_histogram(FAKE, 10, 2, 0, FAKE, FAKE, 1 << 20, None) == -1
    assert lib.foremoe_histogram(FAKE, 10, 2, 8, FAKE, FAKE, 16, None) == -1
    assert b"workspace too small" in lib.foremoe_last_error()
    assert lib.foremoe_histogram(FAKE, 1 << 29, 8, 8, FAKE, FAKE, 1 << 40, None) == -1


def test_assign_rejects_bad_plan(lib):
    from paper_2606_11867_amd._lib import Plan
    p = Plan(8, 4, 0, 0, FAKE, FAKE, FAKE, None, FAKE, FAKE)
    assert lib.foremoe_assign_replicas(FAKE, ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, 1 << 20, None) == -1
    p = Plan(8, 5000, 2, 0, FAKE, FAKE, FAKE, None, FAKE, FAKE)
    assert lib.foremoe_assign_replicas(FAKE, ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, 1 << 20, None) == -1
    assert lib.foremoe_assign_replicas(FAKE, None, FAKE, FAKE, FAKE, FAKE, 1 << 20, None) == -1


def test_histogram_assign_rejects_bad_args(lib):
    from paper_2606_11867_amd._lib import Plan
    p = Plan(8, 4, 2, 0, FAKE, FAKE, FAKE, None, FAKE, FAKE)
    f = lib.foremoe_histogram_assign
    assert f(FAKE, 10, 2, None, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, None) == -1   # no plan
    assert f(None, 10, 2, ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, None) == -1  # no ids
    assert f(FAKE, 10, 0, ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, None) == -1  # K = 0
    assert f(FAKE, 10, 2, ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, FAKE, 16, None) == -1       # small ws
    bad = Plan(8, 4, 0, 0, FAKE, FAKE, FAKE, None, FAKE, FAKE)                                # R_max = 0
    assert f(FAKE, 10, 2, ctypes.byref(bad), FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, None) == -1
    # per-source plan without its source boundaries
    src = Plan(8, 4, 2, 4, FAKE, FAKE, FAKE, None, FAKE, FAKE)
    assert f(FAKE, 10, 2, ctypes.byref(src), FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, None) == -1


def test_permute_rejects_misaligned_rows(lib):
    from paper_2606_11867_amd._lib import Plan
    p = Plan(8, 4, 2, 0, FAKE, FAKE, FAKE, None, FAKE, FAKE)
    rc = lib.foremoe_permute(FAKE, 1, 16, 12, FAKE, 2, ctypes.byref(p), FAKE, FAKE, 32, FAKE, FAKE, FAKE, FAKE,
                             1 << 20, None)
    assert rc == -2  # 12 bf16 elements = 24 bytes, not a multiple of 16


def test_ffn_rejects_unsupported_bf16_shapes(lib):
    rc = lib.foremoe_grouped_ffn_fwd(FAKE, 1, 96, 256, 4, FAKE, FAKE, 3, FAKE, FAKE, 64, FAKE, FAKE, None, None, 0, None)
    assert rc == -2
    rc = lib.foremoe_grouped_ffn_fwd(FAKE, 1, 128, 200, 4, FAKE, FAKE, 3, FAKE, FAKE, 64, FAKE, FAKE, None, None, 0, None)
    assert rc == -2
    rc = lib.foremoe_grouped_ffn_fwd(FAKE, 7, 128, 256, 4, FAKE, FAKE, 3, FAKE, FAKE, 64, FAKE, FAKE, None, None, 0, None)
    assert rc == -1
    rc = lib.foremoe_grouped_ffn_wgrad(FAKE, FAKE, FAKE, FAKE, 1, 128, 128, 4, FAKE, FAKE, 0, 64, FAKE, FAKE,
                                       None, 0, None)
    assert rc == -1  # G < 1
    rc = lib.foremoe_grouped_ffn_wgrad(FAKE, FAKE, FAKE, FAKE, 1, 128, 128, 4, FAKE, FAKE, 2, 64, FAKE, FAKE,
                                       None, 1024, None)
    assert rc == -1  # ws NULL with ws_bytes > 0
    # (n_cap + 256) * row bytes must stay below 4 GiB for 32-bit buffer offsets
    rc = lib.foremoe_grouped_ffn_fwd(FAKE, 1, 8192, 1024, 4, FAKE, FAKE, 3, FAKE, FAKE, 1 << 18, FAKE, FAKE, None,
                                     None, 0, None)
    assert rc == -2
    assert lib.foremoe_wgrad_workspace_size(2048, 768) > 0


def test_ffn_workspace_checks(lib):
    # counters (4 KiB) + one 256 x 256 fp32 partial tile per workgroup of the
    # persistent grid (one per CU; 256 when no device is visible)
    n = lib.foremoe_ffn_workspace_size()
    assert n >= 4096 + 256 * 256 * 4 and (n - 4096) % (256 * 256 * 4) == 0
    args = (FAKE, FAKE, 3, FAKE, FAKE, 64, FAKE, FAKE, None)
    # too small, then misaligned: rejected before any launch
    assert lib.foremoe_grouped_ffn_fwd(FAKE, 1, 128, 256, 4, *args, 1 << 28, n - 1, None) == -1
    assert lib.foremoe_grouped_ffn_fwd(FAKE, 1, 128, 256, 4, *args, (1 << 28) + 16, n, None) == -1
    assert lib.foremoe_grouped_ffn_dgrad(FAKE, FAKE, 1, 128, 256, 4, FAKE, FAKE, 3, FAKE, FAKE, 64, FAKE, FAKE,
                                         1 << 28, 1024, None) == -1


def test_gathers_reject_bad_args(lib):
    assert lib.foremoe_combine(FAKE, 1, FAKE, FAKE, 16, 2, 12, 32, FAKE, 1, None) == -2   # d % 8
    assert lib.foremoe_combine(FAKE, 0, FAKE, FAKE, 16, 2, 16, 32, FAKE, 1, None) == -2   # f32 -> bf16
    assert lib.foremoe_combine(FAKE, 1, FAKE, FAKE, 16, 99, 16, 32, FAKE, 1, None) == -1  # K > 64
    assert lib.foremoe_combine_bwd(FAKE, None, 1, FAKE, FAKE, 16, 2, 16, 32, FAKE, FAKE, None) == -1
    assert lib.foremoe_permute_bwd(FAKE, 1, None, 16, 2, 16, 32, FAKE, 0, None) == -1


def test_empty_calls_launch_nothing(lib):
    # zero tokens: the gathers return before any launch
    assert lib.foremoe_combine(None, 1, None, None, 0, 2, 16, 0, None, 1, None) == 0
    assert lib.foremoe_permute_bwd(None, 1, None, 0, 2, 16, 0, None, 0, None) == 0
    # zero slots: the FFN returns before any launch
    assert lib.foremoe_grouped_ffn_fwd(None, 1, 128, 128, 0, FAKE, None, 1, None, None, 0, None, None, None,
                                       None, 0, None) == 0


def test_bench_refuses_more_than_one_gpu():
    """The benchmark measures one GPU's share; asking for several GPUs ends
    with status 2 and a message, before anything touches a GPU."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"], cwd=root,
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and not r.stdout.strip()


def test_wgrad_steps_check_their_records(lib):
    from paper_2606_11867_amd import _lib
    S = _lib.WgradStep
    ok = S(FAKE, FAKE, FAKE, FAKE, 4, 64)
    one = (S * 1)(ok)
    # bad dtype, shape, G, step count, missing record array: rejected before any launch
    assert lib.foremoe_ffn_gate_up_wgrad_steps(one, 1, 7, 128, 128, 2, 0, 1, FAKE, None, 0, None) == -1
    assert lib.foremoe_ffn_gate_up_wgrad_steps(one, 1, 1, 96, 128, 2, 0, 1, FAKE, None, 0, None) == -2
    assert lib.foremoe_ffn_down_wgrad_steps(one, 1, 1, 128, 128, 0, 0, 1, FAKE, None, 0, None) == -1
    assert lib.foremoe_ffn_down_wgrad_steps(one, _lib.MAX_WGRAD_STEPS + 1, 1, 128, 128, 2, 0, 1, FAKE, None, 0,
                                            None) == -1
    assert lib.foremoe_ffn_down_wgrad_steps(None, 1, 1, 128, 128, 2, 0, 1, FAKE, None, 0, None) == -1
    # the output part must be one of 1..FOREMOE_MAX_WGRAD_STEPS parts
    for part, parts in ((0, 0), (2, 2), (-1, 2), (0, _lib.MAX_WGRAD_STEPS + 1)):
        assert lib.foremoe_ffn_down_wgrad_steps(one, 1, 1, 128, 128, 2, part, parts, FAKE, None, 0, None) == -1
    # a step with a NULL operand, a bad S, a bad n_cap
    for bad in (S(None, FAKE, FAKE, FAKE, 4, 64), S(FAKE, FAKE, FAKE, None, 4, 64), S(FAKE, FAKE, FAKE, FAKE, -1, 64),
                S(FAKE, FAKE, FAKE, FAKE, 4, -5)):
        assert lib.foremoe_ffn_gate_up_wgrad_steps((S * 2)(ok, bad), 2, 1, 128, 128, 2, 0, 1, FAKE, None, 0,
                                                   None) == -1
    # more slots over all steps than one launch can index
    big = S(FAKE, FAKE, FAKE, FAKE, _lib.MAX_SLOTS // 2 + 1, 64)
    assert lib.foremoe_ffn_gate_up_wgrad_steps((S * 2)(big, big), 2, 1, 128, 128, 2, 0, 1, FAKE, None, 0,
                                               None) == -1
    # 32-bit buffer offsets of one step's operands
    assert lib.foremoe_ffn_gate_up_wgrad_steps((S * 1)(S(FAKE, FAKE, FAKE, FAKE, 4, 1 << 21)), 1, 1, 2048, 768, 2,
                                               0, 1, FAKE, None, 0, None) == -2
    # nothing to do (no steps, or only empty ones): returns before any launch, dW untouched
    assert lib.foremoe_ffn_gate_up_wgrad_steps(None, 0, 1, 128, 128, 2, 0, 1, None, None, 0, None) == 0
    empty = (S * 2)(S(None, None, None, None, 0, 64), S(None, None, None, None, 3, 0))
    assert lib.foremoe_ffn_down_wgrad_steps(empty, 2, 1, 128, 128, 2, 0, 1, None, None, 0, None) == 0
