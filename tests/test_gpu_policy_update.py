"""The benchmark's workload end to end at full size: all 16 micro-steps of
the Qwen3-30B-A3B EP=8 rank share in the policy-update stage (T=16384,
d=2048, F=768, E=128, top-8, 16 hosted experts + 4 replica slots per
micro-step), run through the C ABI in exactly the launch configuration the
benchmark times (paper_2606_11867_amd.policy_update: both workspaces, the
weight gradients on a second stream, micro-steps pipelined over two
activation sets). Every micro-step's y, dgates and dx, and the fp32 weight
gradients accumulated over the 16 micro-steps (Sec. 6.2 main-expert
accumulation; App. A.4 fp32 gradients), are compared whole-tensor with the
fp64 oracle: max|err| <= 1e-2 * max|ref| + 1e-3 per tensor."""
import numpy as np
import pytest
import torch

import oracle.foremoe_oracle as O
from tests.gpu_helpers import check_close, config_workload, to_dev, to_np

pytestmark = pytest.mark.gpu


def test_policy_update_full_shape_matches_oracle(gpu):
    from paper_2606_11867_amd import api
    from paper_2606_11867_amd.policy_update import MicroStep, PolicyUpdate
    w = config_workload("qwen3-30b-a3b-ep8-policy-update")
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
                      split=True)
    print(f"\n[case] policy update, {len(mss)} micro-steps, pipelined two-stream schedule, both workspaces",
          flush=True)
    outs = []
    pu.start()
    for i, ms in enumerate(mss):
        pu.run(i, ms, pipelined=True, side_gathers=1)
        st = pu.set_of(i, pipelined=True)
        # copies on the second stream, after permute_bwd (which waited for
        # every main-stream kernel of this micro-step); the set's event is
        # recorded again after them, so micro-step i + 2 reuses the set
        # only once they are done
        with torch.cuda.stream(pu.side):
            outs.append(dict(y=st["y"].clone(), dgates=st["dgates"].clone(), dx=st["dx"].clone(),
                             N=st["slot_offset"][ms.S].clone()))
        pu.done[i % 2].record(pu.side)
    pu.finish()
    torch.cuda.synchronize()
    assert not pu.wws[:256].any().item() and not pu.rws[:4096].any().item(), "workspace counters not reset"

    rgu = np.zeros((G, 2 * F, d))
    rdn = np.zeros((G, d, F))
    Ns = []
    for i, m in enumerate(w.micro):
        fwd = O.layer_forward(w.x(i), m.ids, m.gates, m.plan, gu, dn, n_cap=T * K)
        bwd = O.layer_backward(fwd, w.dy(i), m.gates, m.plan, gu, dn, T, K, rgu, rdn)
        N = int(fwd["slot_offset"][-1])
        Ns.append(N)
        assert int(outs[i]["N"].item()) == N
        print(f"micro-step {i}: N={N}", flush=True)
        check_close(f"y[{i}]", to_np(outs[i]["y"]), fwd["y"])
        check_close(f"dgates[{i}]", to_np(outs[i]["dgates"]), bwd["dgates"])
        check_close(f"dx[{i}]", to_np(outs[i]["dx"]), bwd["dx"])
    # the heaviest micro-steps (about 42k pairs: several full rounds of tiles
    # plus a split tail) are among those checked
    assert max(Ns) > 40000 and min(Ns) < 4000
    check_close("dW_gate_up (16 micro-steps)", to_np(pu.dw_gate_up), rgu)
    check_close("dW_down (16 micro-steps)", to_np(pu.dw_down), rdn)
