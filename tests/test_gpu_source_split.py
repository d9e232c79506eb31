"""GPU parity of the per-source replica split (Sec. 7.2 r_{s,e,j} per source
rank; App. D Stage 4): foremoe_histogram_src, foremoe_assign_replicas and
foremoe_permute with a per-source plan, bit for bit against the oracle.

The planned case takes one rank's share of a micro-step placed by the
planner oracle (Alg. 3: relocation, replication and water-filling over the
8 source ranks of the Qwen3 EP=8 share), whose water-filled token counts
are the per-source weights.
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle.foremoe_oracle as O
import oracle.foremoe_planner as PL
from gpu_helpers import check_close, config_workload, tdtype, to_dev, to_np
from workload import Plan, plan_from_slots

pytestmark = pytest.mark.gpu


def source_loads(ids, E, tb):
    return np.stack([np.bincount(ids[tb[s]:tb[s + 1]].reshape(-1)[ids[tb[s]:tb[s + 1]].reshape(-1) >= 0],
                                 minlength=E) for s in range(len(tb) - 1)]).astype(np.int64)


def planned_share(w, m, rank, N_r=4, C_max=8):
    """Rank `rank`'s slot table for micro-step m, placed by the planner oracle."""
    P, E, T = w.spec.P, w.spec.E, w.spec.T
    tb = np.arange(P + 1, dtype=np.int64) * (T // P)
    loads = [source_loads(mm.ids, E, tb) for mm in w.micro]
    base = PL.base_placement(np.sum(loads, axis=0), 1, P, E // P)
    mp = PL.policy_update_plan(loads[m.index], base, 1, P, E // P, N_r, C_max=C_max)
    mains = [(e, 0) for e in range(E) if mp.copies[e][0] == rank]
    reps = [(e, c) for e in range(E) for c in range(1, len(mp.copies[e])) if mp.copies[e][c] == rank]
    slots = mains + reps
    local = list(dict.fromkeys(e for e, _ in slots))
    widx = np.array([local.index(e) for e, _ in slots], dtype=np.int32)
    plan = Plan(E=E, R_max=C_max, slot_expert=np.array([e for e, _ in slots], np.int32),
                slot_replica=np.array([c for _, c in slots], np.int32),
                expert_nrep=np.array([len(c) for c in mp.copies], np.int32), expert_rep_weight=None,
                slot_widx=widx, slot_gidx=widx.copy(), local_experts=np.array(local, np.int32),
                src_token_begin=tb.astype(np.int32), src_rep_weight=mp.counts.astype(np.int32))
    return plan, mp


def run_both(ids, plan, x, n_cap, dtype, gpu, fused=False):
    from paper_2606_11867_amd import api
    T, K = ids.shape
    tb = plan.src_token_begin
    # oracle
    cs = O.histogram_src(ids, plan.E, tb)
    rb, sc, so = O.assign_replicas_src(cs, plan)
    xp, r2p, p2r, dropped = O.permute_src(x.astype(np.float64), ids, plan, rb, so, n_cap, tb)
    # GPU
    idd = torch.from_numpy(ids).to(gpu)
    dp = api.DevicePlan.from_host(plan, gpu)
    ws = api.workspace(T, K, plan.E * plan.n_src, gpu)
    if fused:  # foremoe_histogram_assign: two launches up to 256 keys, else three
        counts, rep_begin, slot_count, slot_offset = api.histogram_assign(idd, dp, ws)
        counts = counts.reshape(plan.n_src, plan.E)
    else:
        counts = api.histogram_src(idd, plan.E, dp.src_token_begin, ws)
        rep_begin, slot_count, slot_offset = api.assign_replicas(counts.reshape(-1), dp, ws)
    xd = to_dev(x, dtype, gpu)
    x_perm, g_r2p, g_p2r = api.permute(xd, idd, dp, rep_begin, slot_offset, n_cap, ws)
    torch.cuda.synchronize()
    N = int(so[-1])
    assert np.array_equal(counts.cpu().numpy(), cs)
    assert np.array_equal(rep_begin.cpu().numpy(), rb)
    assert np.array_equal(slot_count.cpu().numpy(), sc)
    assert np.array_equal(slot_offset.cpu().numpy(), so)
    assert np.array_equal(g_p2r.cpu().numpy(), p2r)
    M = min(N, n_cap)
    assert np.array_equal(g_r2p.cpu().numpy()[:M], r2p[:M])
    assert np.array_equal(to_np(x_perm[:M]), xp[:M])  # bitwise copies
    status = ws[:256].view(torch.int32).cpu().numpy()
    assert status[1] == dropped and status[2] == 0
    return dict(counts=counts, slot_offset=slot_offset, x_perm=x_perm, pair_to_row=g_p2r, ws=ws,
                ref=dict(so=so, xp=xp, p2r=p2r))


def test_planned_share_bit_exact_and_ffn(gpu):
    from paper_2606_11867_amd import api
    w = config_workload("qwen3-30b-a3b-ep8-share")
    m = w.micro[w.measured]
    plan, mp = planned_share(w, m, rank=w.rank)
    T, K = m.ids.shape
    print(f"planned share: rank {w.rank}, S={plan.S}, copies {[len(c) for c in mp.copies if len(c) > 1]}",
          flush=True)
    x = w.x(m.index)
    got = run_both(m.ids, plan, x, T * K, tdtype(w), gpu, fused=True)  # 1024 keys: three launches
    # the grouped FFN consumes the planned slot table as any other
    N = int(got["ref"]["so"][-1])
    gu, dn = w.weights(plan)
    widx = torch.from_numpy(plan.slot_widx).to(gpu)
    h, y_perm, _ = api.grouped_ffn_fwd(got["x_perm"], got["slot_offset"], widx, to_dev(gu, tdtype(w), gpu),
                                       to_dev(dn, tdtype(w), gpu), save=False)
    torch.cuda.synchronize()
    rows = np.random.default_rng(0).choice(N, size=min(N, 512), replace=False)
    xr = got["ref"]["xp"][rows]
    so = got["ref"]["so"]
    slot = np.searchsorted(so, rows, side="right") - 1
    ref = np.zeros((len(rows), w.spec.d))
    for i, (r, j) in enumerate(zip(rows, slot)):
        g, u = gu[plan.slot_widx[j], :w.spec.F], gu[plan.slot_widx[j], w.spec.F:]
        a, b = g.astype(np.float64) @ xr[i], u.astype(np.float64) @ xr[i]
        ref[i] = dn[plan.slot_widx[j]].astype(np.float64) @ (O.silu(a) * b)
    check_close("y_perm (sampled rows)", to_np(y_perm)[rows], ref)


def natural_share(w, m, rank, C_max=8):
    """Rank `rank`'s slot table for micro-step m under the natural placement
    (expert e on rank e / (E/P), one copy each), written as a per-source
    plan: copy 0 of every expert takes all of its source's pairs."""
    P, E, T = w.spec.P, w.spec.E, w.spec.T
    tb = np.arange(P + 1, dtype=np.int32) * (T // P)
    local = np.arange(rank * (E // P), (rank + 1) * (E // P), dtype=np.int32)
    wts = np.zeros((P, E, C_max), dtype=np.int32)
    wts[:, :, 0] = source_loads(m.ids, E, tb)
    widx = np.arange(len(local), dtype=np.int32)
    return Plan(E=E, R_max=C_max, slot_expert=local, slot_replica=np.zeros(len(local), np.int32),
                expert_nrep=np.ones(E, np.int32), expert_rep_weight=None, slot_widx=widx, slot_gidx=widx.copy(),
                local_experts=local, src_token_begin=tb, src_rep_weight=wts)


@pytest.mark.parametrize("placement", ["natural", "planned"])
def test_slowest_rank_share_bit_exact(gpu, placement):
    """The share of the micro-step's most loaded rank (the one every rank
    waits for, Sec. 7.1 Eq. 1) under either placement: bit-exact dispatch,
    and its local pairs equal to that rank's load."""
    w = config_workload("qwen3-30b-a3b-ep8-share")
    m = w.micro[w.measured]
    P, E, T = w.spec.P, w.spec.E, w.spec.T
    T_, K = m.ids.shape
    if placement == "natural":
        v = m.ids.reshape(-1)
        L = np.bincount(np.arange(E) // (E // P), weights=np.bincount(v[v >= 0], minlength=E), minlength=P)
        rank = int(np.argmax(L))
        plan, load = natural_share(w, m, rank), int(L[rank])
    else:
        tb = np.arange(P + 1, dtype=np.int64) * (T // P)
        loads = [source_loads(mm.ids, E, tb) for mm in w.micro]
        base = PL.base_placement(np.sum(loads, axis=0), 1, P, E // P)
        RL = PL.policy_update_plan(loads[m.index], base, 1, P, E // P, 4, C_max=8).rank_load()
        rank = int(np.argmax(RL))
        plan, _ = planned_share(w, m, rank=rank)
        load = int(RL[rank])
    print(f"{placement} placement: slowest rank {rank}, load {load}, S={plan.S}", flush=True)
    got = run_both(m.ids, plan, w.x(m.index), T_ * K, tdtype(w), gpu, fused=True)
    assert int(got["ref"]["so"][-1]) == load


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_random_sources_bit_exact(gpu, seed):
    rng = np.random.default_rng(seed)
    T, K, E, d = 1500, 3, 9, 64
    ids = rng.integers(0, E, size=(T, K)).astype(np.int32)
    ids[rng.random((T, K)) < 0.1] = -1
    n_src = [2, 5, 8][seed]
    cuts = np.sort(rng.integers(0, T + 1, size=n_src - 1))
    cuts[0] = cuts[1] if n_src > 2 else cuts[0]  # an empty source
    tb = np.concatenate([[0], cuts, [T]]).astype(np.int32)
    plan = plan_from_slots(E, [(2, 0), (0, 0), (0, 2), (5, 1), (7, 0), (0, 1)], nrep={0: 3, 5: 2}, R_max=3)
    wts = rng.integers(0, 5, size=(n_src, E, 3)).astype(np.int32)
    wts[0, 0] = 0  # an all-zero weight row: fine where the block is empty, equal split else
    wts[:, 7] = [1, 0, 0]
    cs = O.histogram_src(ids, E, tb)
    for s in range(n_src):
        for e in range(E):
            if cs[s, e] > 0 and wts[s, e, :plan.expert_nrep[e]].sum() == 0:
                wts[s, e, 0] = 1  # keep the plan error-free
    plan = dataclasses.replace(plan, src_token_begin=tb, src_rep_weight=wts)
    x = rng.standard_normal((T, d)).astype(np.float32)
    N = int(O.assign_replicas_src(cs, plan)[2][-1])
    for n_cap in (N + 3, max(N - 50, 1)):
        for fused in (False, True):
            run_both(ids, plan, x, n_cap, torch.float32, gpu, fused=fused)
