"""Events attached to a row-GEMM launch (foremoe_set_launch_events): they
time the kernel itself, change nothing in its results, and are used once."""
import ctypes

import pytest
import torch

pytestmark = pytest.mark.gpu


def test_launch_events_time_the_kernel(gpu):
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
    for _ in range(2):
        h = torch.zeros(N, F, dtype=bf, device=gpu)
        au = torch.zeros(N, 2 * F, dtype=bf, device=gpu)
        outs.append((h, au))
    call = lambda h, au: lib.foremoe_ffn_gate_up_fwd(  # noqa: E731
        x.data_ptr(), _lib.BF16, d, F, 2, so.data_ptr(), wi.data_ptr(), W, gu.data_ptr(), N,
        h.data_ptr(), au.data_ptr(), None, 0, st.cuda_stream)
    e0, e1, r0, r1 = (torch.cuda.Event(enable_timing=True) for _ in range(4))
    for e in (e0, e1):
        e.record(st)  # create the HIP events
    torch.cuda.synchronize()
    assert call(*outs[0]) == 0  # plain launch
    r0.record(st)
    assert lib.foremoe_set_launch_events(ctypes.c_void_p(e0.cuda_event), ctypes.c_void_p(e1.cuda_event)) == 0
    assert call(*outs[1]) == 0  # launch carrying the events
    r1.record(st)
    torch.cuda.synchronize()
    t_launch, t_bracket = e0.elapsed_time(e1), r0.elapsed_time(r1)
    print(f"kernel {t_launch * 1e3:.1f} us, bracketing records {t_bracket * 1e3:.1f} us", flush=True)
    assert 0.0 < t_launch <= t_bracket * 1.001 + 1e-3
    for a, b in zip(outs[0], outs[1]):
        assert torch.equal(a, b)
    # used once: a further launch leaves the events where they were
    assert call(*outs[1]) == 0
    torch.cuda.synchronize()
    assert e0.elapsed_time(e1) == t_launch
