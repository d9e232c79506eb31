"""The benchmark's workload end to end at full size: all 16 micro-steps of
the Qwen3-30B-A3B EP=8 rank share in the policy-update stage (T=16384,
d=2048, F=768, E=128, top-8, 16 hosted experts + 4 replica slots per
micro-step), run through the C ABI in the launch configurations of
paper_2606_11867_amd.policy_update (both workspaces, micro-steps pipelined):
the weight gradients of every micro-step on a second stream beside its
data-gradient GEMMs; the weight gradients of every group of 8 micro-steps
in one launch pair over the group's rows, on a third stream while the next
group runs; and the benchmark's default: that grouped schedule with each
micro-step's histogram + replica split run on the second stream during the
micro-step before it, and the combine on the second stream. Every
micro-step's y, dgates and dx, and the fp32 weight gradients accumulated over the 16 micro-steps
(Sec. 6.2 main-expert accumulation; App. A.4 fp32 gradients), are compared
whole-tensor with the fp64 oracle: max|err| <= 1e-2 * max|ref| + 1e-3 per
tensor."""
import functools

import numpy as np
import pytest
import torch

import oracle.foremoe_oracle as O
from tests.gpu_helpers import check_close, config_workload, to_dev, to_np

pytestmark = pytest.mark.gpu

NAME = "qwen3-30b-a3b-ep8-policy-update"


@functools.lru_cache(maxsize=None)
def oracle_results():
    """Per micro-step y, dgates, dx, N and the 16-step accumulated gradients."""
    w = config_workload(NAME)
    spec = w.spec
    T, K, F, d = spec.T, spec.K, spec.F, spec.d
    gu, dn = w.weights(w.micro[0].plan)
    G = int(len(w.micro[0].plan.local_experts))
    rgu = np.zeros((G, 2 * F, d))
    rdn = np.zeros((G, d, F))
    per = []
    for i, m in enumerate(w.micro):
        fwd = O.layer_forward(w.x(i), m.ids, m.gates, m.plan, gu, dn, n_cap=T * K)
        bwd = O.layer_backward(fwd, w.dy(i), m.gates, m.plan, gu, dn, T, K, rgu, rdn)
        per.append(dict(y=fwd["y"], dgates=bwd["dgates"], dx=bwd["dx"], N=int(fwd["slot_offset"][-1])))
    return per, rgu, rdn


@pytest.mark.parametrize("wgrad_group,early_hist,side_gathers", [(1, False, 1), (8, False, 1), (8, True, 2)],
                         ids=["wgrad-each", "wgrad-group8", "wgrad-group8-early-hist-combine-side"])
def test_policy_update_full_shape_matches_oracle(gpu, wgrad_group, early_hist, side_gathers):
    from paper_2606_11867_amd import api
    from paper_2606_11867_amd.policy_update import MicroStep, PolicyUpdate
    w = config_workload(NAME)
    spec = w.spec
    T, K, d, F, E = spec.T, spec.K, spec.d, spec.F, spec.E
    bf = torch.bfloat16
    local = w.micro[0].plan.local_experts
    gu, dn = w.weights(w.micro[0].plan)
    G = int(len(local))
    mss = []
    for i, m in enumerate(w.micro):
        assert np.array_equal(m.plan.local_experts, local)
        mss.append(MicroStep(ids=torch.from_numpy(m.ids).to(gpu), gates=torch.from_numpy(m.gates).to(gpu),
                             x=to_dev(w.x(i), bf, gpu), dy=to_dev(w.dy(i), bf, gpu),
                             plan=api.DevicePlan.from_host(m.plan, gpu)))
    pu = PolicyUpdate(T, K, d, F, E, G, max(ms.S for ms in mss), to_dev(gu, bf, gpu), to_dev(dn, bf, gpu), gpu,
                      split=True, wgrad_group=wgrad_group)
    print(f"\n[case] policy update, {len(mss)} micro-steps, pipelined two-stream schedule, both workspaces, "
          f"weight gradients every {wgrad_group} micro-step(s), early histogram {early_hist}, "
          f"second-stream gathers {side_gathers}", flush=True)
    outs = []
    pu.start()
    for i, ms in enumerate(mss):
        nxt = mss[i + 1] if i + 1 < len(mss) else None
        pu.run(i, ms, pipelined=True, side_gathers=side_gathers, next_ms=nxt, early_hist=early_hist)
        st = pu.set_of(i, pipelined=True)
        # copies on the second stream, after permute_bwd (which waited for
        # every main-stream kernel of this micro-step) and the combine; the set's event is
        # recorded again after them, so micro-step i + 2 reuses the set only
        # once they are done
        with torch.cuda.stream(pu.side):
            outs.append(dict(y=st["y"].clone(), dgates=st["dgates"].clone(), dx=st["dx"].clone(),
                             N=st["slot_offset"][ms.S].clone()))
        pu.done[i % 2].record(pu.side)
    pu.finish()
    torch.cuda.synchronize()
    assert not pu.wws[:256].any().item() and not pu.rws[:4096].any().item(), "workspace counters not reset"

    per, rgu, rdn = oracle_results()
    Ns = []
    for i in range(len(w.micro)):
        N = per[i]["N"]
        Ns.append(N)
        assert int(outs[i]["N"].item()) == N
        print(f"micro-step {i}: N={N}", flush=True)
        check_close(f"y[{i}]", to_np(outs[i]["y"]), per[i]["y"])
        check_close(f"dgates[{i}]", to_np(outs[i]["dgates"]), per[i]["dgates"])
        check_close(f"dx[{i}]", to_np(outs[i]["dx"]), per[i]["dx"])
    # the heaviest micro-steps (about 42k pairs: several full rounds of tiles
    # plus a split tail) are among those checked
    assert max(Ns) > 40000 and min(Ns) < 4000
    check_close("dW_gate_up (16 micro-steps)", to_np(pu.dw_gate_up), rgu)
    check_close("dW_down (16 micro-steps)", to_np(pu.dw_down), rdn)


@pytest.mark.parametrize("n_run", [5, 11])
def test_grouped_weight_gradients_flush_an_incomplete_group(gpu, n_run):
    """Micro-steps run in groups of 4 with the two-stream pipelined schedule,
    a number of them that leaves the last group incomplete (finish() then
    launches it): the accumulated gradients equal the oracle's over the
    micro-steps run. Small shapes, several tiles and ragged slots."""
    from paper_2606_11867_amd import api
    from paper_2606_11867_amd.policy_update import MicroStep, PolicyUpdate
    from workload import make_custom
    w = make_custom(T=1024, d=256, F=128, E=32, K=4, P=4, n_rep=2, seed=57, micro_steps=n_run)
    spec = w.spec
    T, K, d, F, E = spec.T, spec.K, spec.d, spec.F, spec.E
    bf = torch.bfloat16
    gu, dn = w.weights(w.micro[0].plan)
    G = int(w.micro[0].plan.G)
    mss = [MicroStep(ids=torch.from_numpy(m.ids).to(gpu), gates=torch.from_numpy(m.gates).to(gpu),
                     x=to_dev(w.x(i), bf, gpu), dy=to_dev(w.dy(i), bf, gpu),
                     plan=api.DevicePlan.from_host(m.plan, gpu)) for i, m in enumerate(w.micro)]
    pu = PolicyUpdate(T, K, d, F, E, G, max(ms.S for ms in mss), to_dev(gu, bf, gpu), to_dev(dn, bf, gpu), gpu,
                      wgrad_group=4)
    print(f"\n[case] {n_run} micro-steps in groups of 4, pipelined", flush=True)
    pu.start()
    for i, ms in enumerate(mss):
        pu.run(i, ms, pipelined=True, side_gathers=1)
    pu.finish()
    torch.cuda.synchronize()
    rgu = np.zeros((G, 2 * F, d))
    rdn = np.zeros((G, d, F))
    for i, m in enumerate(w.micro):
        fwd = O.layer_forward(w.x(i), m.ids, m.gates, m.plan, gu, dn)
        O.layer_backward(fwd, w.dy(i), m.gates, m.plan, gu, dn, T, K, rgu, rdn)
    check_close(f"dW_gate_up ({n_run} micro-steps)", to_np(pu.dw_gate_up), rgu)
    check_close(f"dW_down ({n_run} micro-steps)", to_np(pu.dw_down), rdn)


@pytest.mark.parametrize("wgrad_group", [1, 3])
def test_early_histogram_falls_back_when_inputs_differ(gpu, wgrad_group):
    """The benchmark's schedule (pipelined, combine and the next micro-step's
    histogram + replica split on the second stream) where micro-steps 0 and
    3 announce other inputs for their successor than the ones that then
    run: that successor waits for the early launch and runs its own on the
    main stream; the others announce the right ones. Weight gradients in
    groups of 3 (micro-steps 2 and 5 end a group and launch nothing early)
    or of 1 (each micro-step's own on the second stream, operand sets in a
    ring of 2, every micro-step but the last launches its successor's
    histogram early). Every micro-step's y, dgates and dx and the
    accumulated gradients match the oracle. Small shapes, several tiles and
    ragged slots."""
    from paper_2606_11867_amd import api
    from paper_2606_11867_amd.policy_update import MicroStep, PolicyUpdate
    from workload import make_custom
    w = make_custom(T=1024, d=256, F=128, E=32, K=4, P=4, n_rep=2, seed=61, micro_steps=6)
    spec = w.spec
    T, K, d, F, E = spec.T, spec.K, spec.d, spec.F, spec.E
    bf = torch.bfloat16
    gu, dn = w.weights(w.micro[0].plan)
    G = int(w.micro[0].plan.G)
    mss = [MicroStep(ids=torch.from_numpy(m.ids).to(gpu), gates=torch.from_numpy(m.gates).to(gpu),
                     x=to_dev(w.x(i), bf, gpu), dy=to_dev(w.dy(i), bf, gpu),
                     plan=api.DevicePlan.from_host(m.plan, gpu)) for i, m in enumerate(w.micro)]
    n = len(mss)
    pu = PolicyUpdate(T, K, d, F, E, G, max(ms.S for ms in mss), to_dev(gu, bf, gpu), to_dev(dn, bf, gpu), gpu,
                      wgrad_group=wgrad_group)
    print(f"\n[case] {n} micro-steps, weight gradients in groups of {wgrad_group}, early histogram, wrong "
          "successor announced by micro-steps 0 and 3", flush=True)
    outs = []
    pu.start()
    for i, ms in enumerate(mss):
        nxt = None if i + 1 == n else (mss[(i + 3) % n] if i % 3 == 0 else mss[i + 1])
        if wgrad_group == 3:  # micro-steps 0, 1, 3 and 4 launch their successor's histogram early
            assert pu.wgrad_launches_at(i) == (i % 3 == 2)
        pu.run(i, ms, pipelined=True, side_gathers=2, next_ms=nxt, early_hist=True)
        st = pu.set_of(i, pipelined=True)
        with torch.cuda.stream(pu.side):
            outs.append(dict(y=st["y"].clone(), dgates=st["dgates"].clone(), dx=st["dx"].clone()))
        pu.done[i % 2].record(pu.side)
    pu.finish()
    torch.cuda.synchronize()
    rgu = np.zeros((G, 2 * F, d))
    rdn = np.zeros((G, d, F))
    for i, m in enumerate(w.micro):
        fwd = O.layer_forward(w.x(i), m.ids, m.gates, m.plan, gu, dn)
        bwd = O.layer_backward(fwd, w.dy(i), m.gates, m.plan, gu, dn, T, K, rgu, rdn)
        check_close(f"y[{i}]", to_np(outs[i]["y"]), fwd["y"])
        check_close(f"dgates[{i}]", to_np(outs[i]["dgates"]), bwd["dgates"])
        check_close(f"dx[{i}]", to_np(outs[i]["dx"]), bwd["dx"])
    check_close("dW_gate_up", to_np(pu.dw_gate_up), rgu)
    check_close("dW_down", to_np(pu.dw_down), rdn)


def test_benchmark_dispatch_bit_exact_every_micro_step(gpu):
    """Steps 1-3 of all 16 micro-steps of the benchmark's workload, called as
    the benchmark calls them (foremoe_histogram_assign, then foremoe_permute;
    n_cap = T * K; one workspace reused from micro-step to micro-step, so
    each call starts on what the previous one left): counts, replica bounds,
    slot counts and offsets, both index maps and the permuted rows are
    bit-exact against the oracle (Sec. 5 counts, Sec. 7.2 contiguous replica
    split, Sec. 9 dispatch)."""
    from paper_2606_11867_amd import api
    w = config_workload(NAME)
    T, K = w.micro[0].ids.shape
    n_cap = T * K
    ws = api.workspace(T, K, w.spec.E, gpu)
    for m in w.micro:
        print(f"\n[case] dispatch of micro-step {m.index}", flush=True)
        counts, invalid = O.histogram(m.ids, m.plan.E)
        rb, sc, so = O.assign_replicas(counts, m.plan)
        N = int(so[-1])
        # no pair is dropped at either n_cap, so the maps agree
        xr = w.x(m.index)
        x_perm, r2p, p2r, dropped = O.permute(xr, m.ids, m.plan, rb, so, N + 37)
        assert dropped == 0
        ids = torch.from_numpy(m.ids).to(gpu)
        plan = api.DevicePlan.from_host(m.plan, gpu)
        g_counts, g_rb, g_sc, g_so = api.histogram_assign(ids, plan, ws)
        xd = to_dev(xr, torch.bfloat16, gpu)
        g_xp, g_r2p, g_p2r = api.permute(xd, ids, plan, g_rb, g_so, n_cap, ws)
        torch.cuda.synchronize()
        assert np.array_equal(g_counts.cpu().numpy(), counts)
        assert np.array_equal(g_rb.cpu().numpy(), rb)
        assert np.array_equal(g_sc.cpu().numpy(), sc)
        assert np.array_equal(g_so.cpu().numpy(), so)
        assert np.array_equal(g_p2r.cpu().numpy(), p2r)
        assert np.array_equal(g_r2p.cpu().numpy()[:N], r2p[:N])
        assert np.array_equal(to_np(g_xp[:N]), x_perm[:N])  # bf16 -> f64 is exact
        status = ws[:256].view(torch.int32).cpu().numpy()
        assert status[0] == invalid and status[1] == 0 and status[2] == 0
