"""The transfer engine's one-GPU half on the GPU, through the C ABI, against
the oracle (Sec. 6.1 CPU-assisted prefetch; Sec. 6.2 Copy-out / Copy-in with
main-expert gradient accumulation; App. A.3 records; App. A.4 fp32).

Copy-out and copy-in are copies plus fp32 additions in an order the
interface fixes, so every byte must equal the oracle's. The Qwen3-30B-A3B
expert shape (d=2048, F=768: 27 MiB per record) and a small ragged one are
used; the swap between GPUs is stood in for by a device-to-device copy of
the send buffer."""
import numpy as np
import pytest
import torch

import oracle.foremoe_transfer as X

pytestmark = pytest.mark.gpu


def _host_arrays(W, G, d, F, rng):
    wgu = rng.integers(0, 1 << 16, size=(W, 2 * F, d), dtype=np.uint32).astype(np.uint16)
    wdn = rng.integers(0, 1 << 16, size=(W, d, F), dtype=np.uint32).astype(np.uint16)
    ggu = rng.standard_normal((G, 2 * F, d), dtype=np.float32)
    gdn = rng.standard_normal((G, d, F), dtype=np.float32)
    return wgu, wdn, ggu, gdn


def _dev(arrs, gpu):
    wgu, wdn, ggu, gdn = arrs
    bf = lambda a: torch.from_numpy(a.view(np.int16)).to(gpu).view(torch.bfloat16)  # noqa: E731
    return bf(wgu), bf(wdn), torch.from_numpy(ggu).to(gpu), torch.from_numpy(gdn).to(gpu)


def _back(t):
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


@pytest.mark.parametrize("shape", [(2048, 768, 6, 5), (64, 24, 5, 4)], ids=["qwen3-expert", "small"])
@pytest.mark.parametrize("what", [1, 2, 3], ids=["params", "grads", "both"])
def test_copy_out_bytes(gpu, shape, what):
    from paper_2606_11867_amd import api
    d, F, W, G = shape
    print(f"\n[case] copy_out d={d} F={F} W={W} G={G} what={what}", flush=True)
    rng = np.random.default_rng(10 + what)
    host = _host_arrays(W, G, d, F, rng)
    widx, gidx = [3, 0, 5, 1], [4, 4, 0, 2]
    widx = [w % W for w in widx]
    gidx = [g % G for g in gidx]
    buf = api.copy_out(*_dev(host, gpu), widx, gidx, what)
    torch.cuda.synchronize()
    ref = X.copy_out(*host, widx, gidx, what)
    assert buf.numel() == ref.size
    assert np.array_equal(buf.cpu().numpy(), ref)


@pytest.mark.parametrize("shape", [(2048, 768, 6, 5), (64, 24, 5, 4)], ids=["qwen3-expert", "small"])
def test_copy_in_moves_and_accumulates(gpu, shape):
    """A receive buffer with experts arriving (parameters + assigned
    gradients) and replica partial gradients added into main experts, two of
    them into one target and one after an assign."""
    from paper_2606_11867_amd import api
    d, F, W, G = shape
    print(f"\n[case] copy_in d={d} F={F} W={W} G={G}", flush=True)
    rng = np.random.default_rng(7)
    src = _host_arrays(6, 6, d, F, rng)
    dst = _host_arrays(W, G, d, F, rng)
    what = X.PARAMS | X.GRADS
    buf_h = X.copy_out(*src, list(range(6)), list(range(6)), what)
    widx = [2, -1, -1, 4, -1, 0]
    gidx = [1, 3, 3, 0, 0, -1]
    gmode = [X.ASSIGN, X.ADD, X.ADD, X.ASSIGN, X.ADD, X.ASSIGN]
    ref = X.copy_in(buf_h, widx, gidx, gmode, what, *dst)
    t = _dev(dst, gpu)
    api.copy_in(torch.from_numpy(buf_h).to(gpu), widx, gidx, gmode, what, *t)
    torch.cuda.synchronize()
    for name, got, exp in zip(("w_gate_up", "w_down", "dw_gate_up", "dw_down"), t, ref):
        assert np.array_equal(_back(got).view(np.uint8), np.ascontiguousarray(exp).view(np.uint8)), name


def test_copy_out_swap_copy_in_round_trip(gpu):
    """Copy-out on one expert set, a device-to-device copy standing in for the
    swap, copy-in into another set: the experts arrive bit for bit and every
    replica's partial gradient is summed into its main expert in order."""
    from paper_2606_11867_amd import api
    d, F = 2048, 768
    rng = np.random.default_rng(3)
    a = _host_arrays(4, 4, d, F, rng)
    b = _host_arrays(5, 5, d, F, rng)
    what = X.PARAMS | X.GRADS
    print("\n[case] round trip, 4 Qwen3-shaped experts", flush=True)
    send = api.copy_out(*_dev(a, gpu), [0, 1, 2, 3], [0, 1, 2, 3], what)
    recv = torch.empty_like(send)
    recv.copy_(send)
    tb = _dev(b, gpu)
    widx, gidx, gmode = [4, -1, -1, 1], [4, 2, 2, 1], [X.ASSIGN, X.ADD, X.ADD, X.ASSIGN]
    api.copy_in(recv, widx, gidx, gmode, what, *tb)
    torch.cuda.synchronize()
    ref = X.copy_in(X.copy_out(*a, [0, 1, 2, 3], [0, 1, 2, 3], what), widx, gidx, gmode, what, *b)
    for got, exp in zip(tb, ref):
        assert np.array_equal(_back(got).view(np.uint8), np.ascontiguousarray(exp).view(np.uint8))


def test_prefetch_from_pinned_master(gpu):
    """CPU-assisted prefetch: the C++ plan keeps resident experts, fetches the
    missing ones from the pinned host master copy on a side stream; every
    needed expert then sits in its slot bit for bit."""
    from paper_2606_11867_amd import api
    d, F, E, W = 2048, 768, 16, 6
    print("\n[case] prefetch of Qwen3-shaped experts from pinned host memory", flush=True)
    g = torch.Generator().manual_seed(5)
    master_gu = torch.randn((E, 2 * F, d), generator=g).to(torch.bfloat16).pin_memory()
    master_dn = torch.randn((E, d, F), generator=g).to(torch.bfloat16).pin_memory()
    resident = [3, 7, -1, 5, 11, 2]
    wgu = torch.zeros((W, 2 * F, d), dtype=torch.bfloat16, device=gpu)
    wdn = torch.zeros((W, d, F), dtype=torch.bfloat16, device=gpu)
    for w, e in enumerate(resident):
        if e >= 0:
            wgu[w].copy_(master_gu[e])
            wdn[w].copy_(master_dn[e])
    torch.cuda.synchronize()
    needed = [5, 2, 3, 9, 14]
    slot_of, fe, fw = api.plan_prefetch(resident, needed)
    so_o, f_o = X.plan_prefetch(resident, needed)
    assert slot_of.tolist() == so_o and list(zip(fe.tolist(), fw.tolist())) == f_o
    side = torch.cuda.Stream(gpu)
    side.wait_stream(torch.cuda.current_stream(gpu))
    api.prefetch_experts(master_gu, master_dn, fe, fw, wgu, wdn, stream=side)
    torch.cuda.current_stream(gpu).wait_stream(side)
    torch.cuda.synchronize()
    for e, w in zip(needed, slot_of.tolist()):
        assert torch.equal(wgu[w].cpu(), master_gu[e]) and torch.equal(wdn[w].cpu(), master_dn[e]), (e, w)
