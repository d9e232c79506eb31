"""Timed row-GEMM calls (foremoe_ffn_*_timed): the events time the kernel
itself, the results equal the plain call's, and nothing is left attached
for a later call."""
import ctypes

import pytest
import torch

pytestmark = pytest.mark.gpu


def test_timed_call_times_the_kernel(gpu):
    from paper_2606_11867_amd import _lib
    lib = _lib.load()
    d, F, N, W = 2048, 768, 8192, 2
    g = torch.Generator(device="cpu").manual_seed(3)
    bf = torch.bfloat16
    x = torch.randn(N, d, generator=g).to(bf).to(gpu)
    gu = (torch.randn(W, 2 * F, d, generator=g) / d ** 0.5).to(bf).to(gpu)
    so = torch.tensor([0, 5000, N], dtype=torch.int32, device=gpu)
    wi = torch.tensor([0, 1], dtype=torch.int32, device=gpu)
    st = torch.cuda.current_stream(gpu)
    outs = []
    for _ in range(3):
        h = torch.zeros(N, F, dtype=bf, device=gpu)
        au = torch.zeros(N, 2 * F, dtype=bf, device=gpu)
        outs.append((h, au))
    args = lambda h, au: (x.data_ptr(), _lib.BF16, d, F, 2, so.data_ptr(), wi.data_ptr(), W,  # noqa: E731
                          gu.data_ptr(), N, h.data_ptr(), au.data_ptr(), None, 0, st.cuda_stream)
    e0, e1, r0, r1 = (torch.cuda.Event(enable_timing=True) for _ in range(4))
    for e in (e0, e1):
        e.record(st)  # create the HIP events
    torch.cuda.synchronize()
    print("[case] gate/up forward, 2 slots, N=8192, plain then timed then plain", flush=True)
    assert lib.foremoe_ffn_gate_up_fwd(*args(*outs[0])) == 0
    r0.record(st)
    assert lib.foremoe_ffn_gate_up_fwd_timed(*args(*outs[1]), ctypes.c_void_p(e0.cuda_event),
                                             ctypes.c_void_p(e1.cuda_event)) == 0
    r1.record(st)
    torch.cuda.synchronize()
    t_launch, t_bracket = e0.elapsed_time(e1), r0.elapsed_time(r1)
    print(f"kernel {t_launch * 1e3:.1f} us, bracketing records {t_bracket * 1e3:.1f} us", flush=True)
    assert 0.0 < t_launch <= t_bracket * 1.001 + 1e-3
    # a later plain call does not touch the events
    assert lib.foremoe_ffn_gate_up_fwd(*args(*outs[2])) == 0
    torch.cuda.synchronize()
    assert e0.elapsed_time(e1) == t_launch
    for o in outs[1:]:
        for a, b in zip(outs[0], o):
            assert torch.equal(a, b)


def test_timed_call_without_work_records_both_events(gpu):
    from paper_2606_11867_amd import _lib
    lib = _lib.load()
    st = torch.cuda.current_stream(gpu)
    e0, e1 = (torch.cuda.Event(enable_timing=True) for _ in range(2))
    so = torch.zeros(1, dtype=torch.int32, device=gpu)
    # first records around a long fill (this also creates the HIP events,
    # which torch makes on first record): their elapsed time covers the fill
    big = torch.empty(1 << 30, dtype=torch.uint8, device=gpu)
    e0.record(st)
    big.fill_(1)
    e1.record(st)
    torch.cuda.synchronize()
    t_fill = e0.elapsed_time(e1)
    assert t_fill > 0.05
    print("[case] down forward with S=0 (nothing launched), timed", flush=True)
    assert lib.foremoe_ffn_down_fwd_timed(None, _lib.BF16, 256, 256, 0, so.data_ptr(), None, 1, None, 0, None,
                                          None, 0, st.cuda_stream, ctypes.c_void_p(e0.cuda_event),
                                          ctypes.c_void_p(e1.cuda_event)) == 0
    torch.cuda.synchronize()
    assert e0.query() and e1.query()
    assert 0.0 <= e0.elapsed_time(e1) < 0.05
