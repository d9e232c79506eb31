"""Weight gradients of several micro-steps in one call
(foremoe_ffn_{gate_up,down}_wgrad_steps) against the fp64 oracle: the sum
over the micro-steps of each one's main-expert gradients (Sec. 6.2), added
in fp32 onto a non-zero start (App. A.4). Each micro-step has its own
routing, slot table and replica choice; operand buffers have more rows than
the slots cover, and the rows past the last slot hold garbage that must not
be read. Tolerance: max|err| <= 1e-2 * max|ref| + 1e-3 per tensor."""
import numpy as np
import pytest
import torch

import oracle.foremoe_oracle as O
from tests.gpu_helpers import check_close, custom_workload, oracle_dispatch, rnd, tdtype, to_dev, to_np

pytestmark = pytest.mark.gpu


def _operands(w, m, rng):
    """One micro-step's weight-gradient operands (rounded to the storage
    precision), from the oracle's dispatch, forward and dgrad."""
    ref = oracle_dispatch(w, m)
    N = int(ref["slot_offset"][-1])
    gu, dn = w.weights(m.plan)
    x_perm = ref["x_perm"][:N]
    F, d = w.spec.F, w.spec.d
    f = O.ffn_forward(x_perm, ref["slot_offset"], m.plan.slot_widx, gu, dn)
    dy_perm = rnd(w, rng.standard_normal((N, d)))
    hq = rnd(w, f["H"])
    g = O.ffn_dgrad(dy_perm, rnd(w, f["A"]), rnd(w, f["U"]), ref["slot_offset"], m.plan.slot_widx, gu, dn)
    dau = rnd(w, np.concatenate([g["dA"], g["dU"]], axis=1))
    return dict(x_perm=x_perm, h=hq, dy_perm=dy_perm, d_au=dau, slot_offset=ref["slot_offset"],
                slot_gidx=m.plan.slot_gidx, N=N)


def _to_gpu(op, w, gpu, pad, rng):
    """Device copies with `pad` extra rows of garbage past the last slot."""
    dt = tdtype(w)
    out = {}
    for k in ("x_perm", "h", "dy_perm", "d_au"):
        a = op[k]
        junk = rng.standard_normal((pad, a.shape[1])) * 1e3
        out[k] = to_dev(np.concatenate([a, junk], axis=0), dt, gpu)
    out["slot_offset"] = torch.from_numpy(np.ascontiguousarray(op["slot_offset"], dtype=np.int32)).to(gpu)
    out["slot_gidx"] = torch.from_numpy(np.ascontiguousarray(op["slot_gidx"], dtype=np.int32)).to(gpu)
    return out


@pytest.mark.parametrize("ws_kind", ["none", "counters", "split"])
@pytest.mark.parametrize("name", ["share", "small", "tinyf32"])
def test_wgrad_steps_matches_oracle(gpu, name, ws_kind):
    from paper_2606_11867_amd import api
    w = custom_workload(name)
    rng = np.random.default_rng(91)
    # several micro-steps with different routing; a workload with one
    # micro-step contributes it twice (the sum must then double)
    idx = list(range(len(w.micro))) if len(w.micro) > 1 else [0, 0]
    ops = [_operands(w, w.micro[i], rng) for i in idx]
    G = w.micro[0].plan.G
    d, F = w.spec.d, w.spec.F
    print(f"\n[case] {name}: {len(ops)} micro-steps, N={[o['N'] for o in ops]}, G={G}, workspace {ws_kind}",
          flush=True)
    start_gu = rng.standard_normal((G, 2 * F, d)).astype(np.float32)
    start_dn = rng.standard_normal((G, d, F)).astype(np.float32)
    rgu, rdn = start_gu.astype(np.float64), start_dn.astype(np.float64)
    for o in ops:
        rgu, rdn = O.ffn_wgrad(o["x_perm"], o["h"], o["dy_perm"], o["d_au"][:, :F], o["d_au"][:, F:],
                               o["slot_offset"], o["slot_gidx"], G, rgu, rdn)
    steps = [_to_gpu(o, w, gpu, pad=37, rng=rng) for o in ops]
    ws = {"none": None, "counters": torch.zeros(256, dtype=torch.uint8, device=gpu),
          "split": api.wgrad_workspace(d, F, gpu)}[ws_kind]
    dwgu = torch.from_numpy(start_gu.copy()).to(gpu)
    dwdn = torch.from_numpy(start_dn.copy()).to(gpu)
    api.grouped_ffn_wgrad_steps(steps, dwgu, dwdn, ws=ws)
    torch.cuda.synchronize()
    check_close("dW_gate_up (steps)", to_np(dwgu), rgu)
    check_close("dW_down (steps)", to_np(dwdn), rdn)
    if ws is not None:
        assert not ws[:256].any().item(), "work counters not reset"
    # the same gradients as one call per micro-step (up to fp32 rounding)
    one_gu = torch.from_numpy(start_gu.copy()).to(gpu)
    one_dn = torch.from_numpy(start_dn.copy()).to(gpu)
    for st in steps:
        api.grouped_ffn_wgrad(st["x_perm"], st["h"], st["dy_perm"], st["d_au"], st["slot_offset"],
                              st["slot_gidx"], one_gu, one_dn, ws=ws)
    torch.cuda.synchronize()
    check_close("steps vs per-micro-step calls (gate/up)", to_np(dwgu), to_np(one_gu))
    check_close("steps vs per-micro-step calls (down)", to_np(dwdn), to_np(one_dn))


def test_wgrad_steps_deterministic_and_skips_empty(gpu):
    """Repeated calls give bit-identical results; a micro-step with no slots
    and an empty step list change nothing."""
    from paper_2606_11867_amd import _lib, api
    w = custom_workload("share")
    rng = np.random.default_rng(92)
    ops = [_operands(w, m, rng) for m in w.micro]
    G, d, F = w.micro[0].plan.G, w.spec.d, w.spec.F
    steps = [_to_gpu(o, w, gpu, pad=5, rng=rng) for o in ops]
    ws = api.wgrad_workspace(d, F, gpu)
    outs = []
    for _ in range(2):
        dwgu = torch.zeros((G, 2 * F, d), dtype=torch.float32, device=gpu)
        dwdn = torch.zeros((G, d, F), dtype=torch.float32, device=gpu)
        api.grouped_ffn_wgrad_steps(steps, dwgu, dwdn, ws=ws)
        torch.cuda.synchronize()
        outs.append((dwgu.clone(), dwdn.clone()))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])
    # an extra micro-step with S = 0 (its pointers are never read) and a call with no steps
    lib = _lib.load()
    arr = api.wgrad_steps(steps, a="d_au", b="x_perm")
    ext = (_lib.WgradStep * (len(steps) + 1))(*list(arr), _lib.WgradStep(None, None, None, None, 0, 0))
    dwgu = torch.zeros((G, 2 * F, d), dtype=torch.float32, device=gpu)
    st = torch.cuda.current_stream().cuda_stream
    assert lib.foremoe_ffn_gate_up_wgrad_steps(ext, len(steps) + 1, _lib.BF16, d, F, G, 0, 1, dwgu.data_ptr(),
                                               ws.data_ptr(), ws.numel(), st) == 0
    assert lib.foremoe_ffn_gate_up_wgrad_steps(ext, 0, _lib.BF16, d, F, G, 0, 1, dwgu.data_ptr(),
                                               ws.data_ptr(), ws.numel(), st) == 0
    torch.cuda.synchronize()
    assert torch.equal(dwgu, outs[0][0])


@pytest.mark.parametrize("parts", [2, 3, 4])
def test_wgrad_steps_parts_cover_the_tiles(gpu, parts):
    """The parts of one group of micro-steps, launched one after another,
    give the whole update; a part touches only its own output tiles (256 x
    256 tiles for dW_gate_up [768, 512], 128 x 128 for dW_down [512, 384])."""
    from paper_2606_11867_amd import api
    from workload import make_custom
    w = make_custom(T=1024, d=512, F=384, E=16, K=2, P=2, n_rep=2, seed=93, micro_steps=3)
    rng = np.random.default_rng(94)
    ops = [_operands(w, m, rng) for m in w.micro]
    G, d, F = w.micro[0].plan.G, w.spec.d, w.spec.F
    print(f"\n[case] parts={parts}: {len(ops)} micro-steps, N={[o['N'] for o in ops]}, G={G}", flush=True)
    start_gu = rng.standard_normal((G, 2 * F, d)).astype(np.float32)
    start_dn = rng.standard_normal((G, d, F)).astype(np.float32)
    rgu, rdn = start_gu.astype(np.float64), start_dn.astype(np.float64)
    for o in ops:
        rgu, rdn = O.ffn_wgrad(o["x_perm"], o["h"], o["dy_perm"], o["d_au"][:, :F], o["d_au"][:, F:],
                               o["slot_offset"], o["slot_gidx"], G, rgu, rdn)
    steps = [_to_gpu(o, w, gpu, pad=11, rng=rng) for o in ops]
    ws = api.wgrad_workspace(d, F, gpu)
    dwgu = torch.from_numpy(start_gu.copy()).to(gpu)
    dwdn = torch.from_numpy(start_dn.copy()).to(gpu)

    def tile_mask(M, N, bm, bn, part):
        t = (np.arange(M)[:, None] // bm) * (N // bn) + np.arange(N)[None, :] // bn
        return (t % parts) == part

    for part in range(parts):
        api.grouped_ffn_wgrad_steps(steps, dwgu, dwdn, ws=ws, part=part, parts=parts)
        torch.cuda.synchronize()
        if part == 0:
            # only part 0's tiles have moved
            mgu = tile_mask(2 * F, d, 256, 256, 0)
            mdn = tile_mask(d, F, 128, 128, 0)
            gu0, dn0 = to_np(dwgu), to_np(dwdn)
            assert np.array_equal(gu0[:, ~mgu], start_gu[:, ~mgu].astype(np.float64))
            assert np.array_equal(dn0[:, ~mdn], start_dn[:, ~mdn].astype(np.float64))
            assert not np.array_equal(gu0[:, mgu], start_gu[:, mgu].astype(np.float64))
    check_close(f"dW_gate_up ({parts} parts)", to_np(dwgu), rgu)
    check_close(f"dW_down ({parts} parts)", to_np(dwdn), rdn)
    assert not ws[:256].any().item(), "work counters not reset"
