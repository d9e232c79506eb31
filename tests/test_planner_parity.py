"""The C++ planner (foremoe_plan_*) against the planner oracle, bit for bit.

Host-only: the planner runs on the CPU, so these tests need the built
library but no GPU.
"""
import numpy as np
import pytest

import oracle.foremoe_planner as PL
from workload import make_workload


@pytest.fixture(scope="module")
def api():
    import os
    import paper_2606_11867_amd as fm
    if not os.path.exists(fm.LIB_PATH):
        from paper_2606_11867_amd import build
        build.build()
    from paper_2606_11867_amd import api
    return api


def oracle_arrays(mp, C_max):
    E = mp.E
    cr = np.full((E, C_max), -1, dtype=np.int64)
    for e, c in enumerate(mp.copies):
        cr[e, :len(c)] = c
    counts = np.zeros((mp.P, E, C_max), dtype=np.int64)
    counts[:, :, :mp.counts.shape[2]] = mp.counts
    return cr, counts


def compare(api, w, M, R, N_b, N_r, c_load=1, c_traffic=0, C_max=8):
    w = np.asarray(w, dtype=np.int64)
    base_o = PL.base_placement(w, M, R, N_b, c_load, c_traffic)
    base_g = api.plan_base(w, M, R, N_b, c_load, c_traffic)
    assert base_g.tolist() == base_o.tolist()
    mp = PL.policy_update_plan(w, base_o, M, R, N_b, N_r)
    cr_o, cnt_o = oracle_arrays(mp, C_max)
    cr_g, cnt_g, load_g = api.plan_micro_step(w, base_g, M, R, N_b, N_r, C_max)
    assert np.array_equal(cr_g, cr_o)
    assert np.array_equal(cnt_g, cnt_o)
    assert load_g.tolist() == mp.rank_load().tolist()
    return mp, cr_g


def test_worked_water_filling_case(api):
    compare(api, [[60, 10], [40, 0]], M=1, R=2, N_b=1, N_r=1)


def test_worked_stage_cases(api):
    # the hand-worked Stage 2, Stage 3-4 and machine-confinement cases of the
    # planner pins, through the C++ planner
    for w, M, R, N_b, N_r, base in (
            ([[10, 9, 1, 1], [0, 0, 0, 0]], 1, 2, 2, 0, [0, 0, 1, 1]),
            ([[100, 90, 70, 10], [0] * 4, [0] * 4, [0] * 4], 1, 4, 1, 1, [0, 1, 2, 3]),
            ([[500, 10, 0, 0], [0] * 4, [0] * 4, [0] * 4], 2, 2, 1, 1, [0, 1, 2, 3])):
        w = np.asarray(w, dtype=np.int64)
        mp = PL.policy_update_plan(w, np.asarray(base), M, R, N_b, N_r)
        cr_o, cnt_o = oracle_arrays(mp, 8)
        cr_g, cnt_g, load_g = api.plan_micro_step(w, np.asarray(base), M, R, N_b, N_r, 8)
        assert np.array_equal(cr_g, cr_o) and np.array_equal(cnt_g, cnt_o)
        assert load_g.tolist() == mp.rank_load().tolist()


@pytest.mark.parametrize("seed", range(6))
def test_random_machines(api, seed):
    rng = np.random.default_rng(seed)
    M, R = int(rng.integers(1, 4)), int(rng.integers(1, 5))
    N_b, N_r = int(rng.integers(1, 4)), int(rng.integers(0, 3))
    P = M * R
    E = int(rng.integers(1, P * N_b + 1))
    w = (rng.pareto(1.1, size=(P, E)) * rng.integers(1, 40)).astype(np.int64)
    w[rng.random((P, E)) < 0.2] = 0
    compare(api, w, M, R, N_b, N_r, c_load=int(rng.integers(0, 5)), c_traffic=int(rng.integers(0, 5)))


def source_loads(w, m):
    P, E, T = w.spec.P, w.spec.E, w.spec.T
    src = np.repeat(np.arange(P), T // P)
    return np.stack([np.bincount(m.ids[src == s].reshape(-1), minlength=E) for s in range(P)]).astype(np.int64)


def test_policy_update_workload(api):
    # the Qwen3 EP=8 share: one machine of 8 ranks, 16 base + 4 redundant
    # slots per rank; every micro-step planned by both and compared
    w = make_workload("qwen3-30b-a3b-ep8-policy-update")
    P, E = w.spec.P, w.spec.E
    loads = [source_loads(w, m) for m in w.micro]
    agg = np.sum(loads, axis=0)
    base = api.plan_base(agg, 1, P, E // P)
    assert base.tolist() == PL.base_placement(agg, 1, P, E // P).tolist()
    for W in loads[:4]:
        mp = PL.policy_update_plan(W, base, 1, P, E // P, 4)
        cr_o, cnt_o = oracle_arrays(mp, 8)
        cr_g, cnt_g, load_g = api.plan_micro_step(W, base, 1, P, E // P, 4, 8)
        assert np.array_equal(cr_g, cr_o) and np.array_equal(cnt_g, cnt_o)
        assert load_g.tolist() == mp.rank_load().tolist()


def test_rank_slots(api):
    rng = np.random.default_rng(9)
    M, R, N_b, N_r = 1, 4, 3, 2
    w = (rng.pareto(1.0, size=(4, 12)) * 30).astype(np.int64)
    mp, cr = compare(api, w, M, R, N_b, N_r)
    for rank in range(M * R):
        got = api.plan_rank_slots(cr, rank)
        mains = [(e, 0) for e in range(12) if mp.copies[e][0] == rank]
        reps = [(e, c) for e in range(12) for c in range(1, len(mp.copies[e])) if mp.copies[e][c] == rank]
        slots = mains + reps
        assert list(zip(got["slot_expert"].tolist(), got["slot_replica"].tolist())) == slots
        local = list(dict.fromkeys(e for e, _ in slots))
        assert got["local_experts"].tolist() == local
        assert got["slot_widx"].tolist() == [local.index(e) for e, _ in slots]
        assert got["expert_nrep"].tolist() == [len(c) for c in mp.copies]


def test_errors(api):
    from paper_2606_11867_amd._lib import ForeMoEError
    w = np.array([[100, 5], [100, 5]])
    with pytest.raises(ForeMoEError):
        api.plan_micro_step(w, np.array([0, 1]), 1, 2, 1, 1, C_max=1)  # needs 2 copies
    with pytest.raises(ForeMoEError):
        api.plan_base(np.ones((2, 5)), 1, 2, 2)  # 5 experts, 4 base slots
    with pytest.raises(ForeMoEError):
        api.plan_base(-np.ones((2, 2)), 1, 2, 1)
