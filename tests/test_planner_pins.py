"""Pins of the planner oracle (Sec. 8, Alg. 1; App. D, Alg. 3).

Independent formulations only: hand-worked LPT and water-filling cases
(derived step by step in the comments), Graham's list-scheduling bound,
the constraints of the placement (token conservation and feasibility,
Sec. 7.2 and App. C; slot capacities), and the closed-form water level of a
single replicated expert. Mutation tests plant plausible mistakes in the
oracle (on the CPU) and require a pin to catch them.
"""
import numpy as np
import pytest

import oracle.foremoe_planner as PL


# ---------------------------------------------------------------------------
# LPT (Alg. 1 rank level; Alg. 3 Stage 2)
# ---------------------------------------------------------------------------
def check_lpt_textbook():
    # loads 7,6,5,4,3 on two ranks: 7->r0, 6->r1, 5->r1 (6 < 7), 4->r0
    # (7 < 11), 3 -> tie 11/11 -> lower rank r0: loads 14 / 11
    w = np.array([7, 6, 5, 4, 3])
    got = PL.rank_lpt(w, range(5), [0, 1], cap=5)
    return got == {0: 0, 1: 1, 2: 1, 3: 0, 4: 0}


def check_lpt_graham(seed=0):
    rng = np.random.default_rng(seed)
    for _ in range(20):
        n, R = int(rng.integers(1, 40)), int(rng.integers(1, 9))
        w = rng.integers(0, 1000, size=n)
        got = PL.rank_lpt(w, range(n), list(range(R)), cap=n)
        if sorted(got) != list(range(n)):
            return False
        load = np.bincount([got[e] for e in range(n)], weights=w, minlength=R)
        # list scheduling: makespan <= total / R + largest job
        if load.max() > w.sum() / R + w.max() + 1e-9:
            return False
    return True


def test_lpt_textbook():
    assert check_lpt_textbook()


def test_lpt_graham_bound():
    assert check_lpt_graham()


def test_lpt_capacity():
    # one dominant expert cannot pull two experts onto the empty rank past
    # its capacity: with cap 2 on 2 ranks, loads 100,1,1,1 -> the three
    # light experts fill r1 (cap 2) and then r0
    got = PL.rank_lpt(np.array([100, 1, 1, 1]), range(4), [0, 1], cap=2)
    counts = np.bincount(list(got.values()), minlength=2)
    assert counts.tolist() == [2, 2] and got[0] == 0


# ---------------------------------------------------------------------------
# Stage 1 machine level (Alg. 1)
# ---------------------------------------------------------------------------
def test_base_traffic_only_keeps_experts_near_their_sources():
    # two machines of one rank each; experts 0, 1 are loaded only from
    # source 0 (machine 0), experts 2, 3 only from source 1: with the
    # traffic term alone every expert lands where its tokens come from
    w = np.array([[9, 8, 0, 0], [0, 0, 7, 6]])
    rank = PL.base_placement(w, M=2, R=1, N_b=2, c_load=0, c_traffic=1)
    assert rank.tolist() == [0, 0, 1, 1]


def test_base_load_only_balances_machines():
    # load term alone, machines of 2 ranks x 2 slots: aggregate loads
    # 10, 9, 2, 1 (ties none). Machine level: 10 -> m0, 9 -> m1, 2 -> m1
    # (9 < 10), 1 -> m0 (10 < 11). Rank level on m0 (ranks 0, 1): 10 -> r0,
    # 1 -> r1; on m1 (ranks 2, 3): 9 -> r2, 2 -> r3.
    w = np.array([[5, 4, 1, 1], [5, 5, 1, 0], [0, 0, 0, 0], [0, 0, 0, 0]])
    rank = PL.base_placement(w, M=2, R=2, N_b=2, c_load=1, c_traffic=0)
    assert rank.tolist() == [0, 2, 3, 1]


# ---------------------------------------------------------------------------
# Stages 2-4 (Alg. 3)
# ---------------------------------------------------------------------------
def check_water_filling_worked_example():
    # two ranks, one base slot and one redundant slot each. e0 has 60 tokens
    # from source 0 and 40 from source 1, e1 has 10 from source 0.
    # Stage 2: e0 -> r0, e1 -> r1. Stage 3: e0 is heaviest, r1 has the
    # least load and no copy of e0 -> replica of e0 on r1; the second round
    # picks e0 again (50 per copy > 10) but no rank can take it -> stop.
    # Stage 4: r1 starts at 10 (e1), r0 at 0. Source 0: the first 10 units
    # go to r0 (loads 10 / 10), then ties go to copy 0 first, so the other
    # 50 alternate 25 / 25 -> c[0][e0] = (35, 25), loads 35 / 35; source 1
    # alternates from copy 0: (20, 20).
    w = np.array([[60, 10], [40, 0]])
    mp = PL.policy_update_plan(w, np.array([0, 1]), M=1, R=2, N_b=1, N_r=1)
    return (mp.copies == [[0, 1], [1]] and mp.counts[0, 0].tolist() == [35, 25]
            and mp.counts[1, 0].tolist() == [20, 20] and mp.counts[0, 1, 0] == 10
            and mp.rank_load().tolist() == [55, 55])


def test_water_filling_worked_example():
    assert check_water_filling_worked_example()


def water_level_counts(base_loads, n):
    """Closed form: fill bins of initial levels base_loads with n units, one
    at a time onto the lowest level (lowest index among equals)."""
    L = np.asarray(base_loads, dtype=np.int64)
    lo, hi = int(L.min()), int(L.max()) + n + 1
    while lo < hi:  # largest level lam with sum(max(0, lam - L)) <= n
        mid = (lo + hi + 1) // 2
        if np.maximum(0, mid - L).sum() <= n:
            lo = mid
        else:
            hi = mid - 1
    c = np.maximum(0, lo - L)
    rest = n - int(c.sum())
    for i in np.nonzero(L <= lo)[0][:rest]:  # bins now at level lo, in index order
        c[i] += 1
    return c


def check_single_replica_water_level(seed=1):
    rng = np.random.default_rng(seed)
    for _ in range(10):
        # one machine of 4 ranks, 4 experts on 4 base slots, exactly one
        # expert heavy enough to take every replica slot (N_r = 1 -> a copy
        # of expert 0 on every rank)
        P = 4
        w = rng.integers(0, 30, size=(P, 4))
        w[:, 0] = rng.integers(200, 400, size=P)
        mp = PL.policy_update_plan(w, np.array([0, 1, 2, 3]), M=1, R=P, N_b=1, N_r=1)
        if sorted(mp.copies[0]) != [0, 1, 2, 3] or any(len(mp.copies[e]) != 1 for e in range(1, 4)):
            return False
        # initial levels: each rank's non-replicated expert
        base = np.zeros(P, dtype=np.int64)
        for e in range(1, 4):
            base[mp.copies[e][0]] += w[:, e].sum()
        lv = base[mp.copies[0]]
        if mp.counts[:, 0, :].sum(axis=0).tolist() != water_level_counts(lv, int(w[:, 0].sum())).tolist():
            return False
    return True


def test_single_replica_water_level():
    assert check_single_replica_water_level()


def check_plan_constraints(mp, w, M, R, N_b, N_r):
    P, E = w.shape
    # token conservation: sum over copies of r_{s,e,j} w_{s,e} = w_{s,e}
    if not np.array_equal(mp.counts.sum(axis=2), w):
        return False
    base = np.zeros(P, int)
    reps = np.zeros(P, int)
    for e in range(E):
        c = mp.copies[e]
        if len(set(c)) != len(c) or len({r // R for r in c}) != 1:
            return False  # two copies on one rank, or a cross-machine replica
        base[c[0]] += 1
        for r in c[1:]:
            reps[r] += 1
        # feasibility: no tokens for copies that do not exist
        if mp.counts[:, e, len(c):].any():
            return False
    return bool((base <= N_b).all() and (reps <= N_r).all())


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_plan_constraints_random(seed):
    rng = np.random.default_rng(seed)
    M, R, N_b, N_r = 2, 4, 3, 1
    P, E = M * R, M * R * N_b
    w = (rng.pareto(1.2, size=(P, E)) * 20).astype(np.int64)
    base = PL.base_placement(w, M, R, N_b, c_load=3, c_traffic=1)
    mp = PL.policy_update_plan(w, base, M, R, N_b, N_r)
    assert check_plan_constraints(mp, w, M, R, N_b, N_r)
    assert mp.rank_load().sum() == w.sum()


def test_policy_update_lowers_imbalance_on_generated_routing():
    # the Qwen3 EP=8 share's micro-steps: the planned rank loads are better
    # balanced than the base placement's in the median (the paper reports
    # the same direction, Sec. 10.4)
    from workload import make_workload
    w = make_workload("qwen3-30b-a3b-ep8-policy-update")
    P, E, T = w.spec.P, w.spec.E, w.spec.T
    loads = []
    for m in w.micro[:6]:
        src = np.repeat(np.arange(P), T // P)
        W = np.stack([np.bincount(m.ids[src == s].reshape(-1), minlength=E) for s in range(P)])
        loads.append(W.astype(np.int64))
    base = PL.base_placement(np.sum(loads, axis=0), 1, P, E // P)
    before, after = [], []
    for W in loads:
        mp = PL.policy_update_plan(W, base, 1, P, E // P, 4)
        assert check_plan_constraints(mp, W, 1, P, E // P, 4)
        before.append(PL.imbalance(np.bincount(base, weights=W.sum(0), minlength=P)))
        after.append(PL.imbalance(mp.rank_load()))
    assert np.median(after) < np.median(before)


# ---------------------------------------------------------------------------
# Hand-worked cases that tell the App. D rules apart
# ---------------------------------------------------------------------------
def check_stage2_relocation():
    # One machine of two ranks with two base slots each; all tokens come
    # from source 0. The base placement (from the aggregate) put e0, e1 on r0
    # and e2, e3 on r1, but this micro-step's loads are 10, 9, 1, 1.
    # Stage 2 (LPT on the micro-step load): e0 (10) -> r0 (0/0, lower id);
    # e1 (9) -> r1 (0 < 10); e2 (1) -> r1 (9 < 10); e3 (1) -> tie 10/10 ->
    # r0. Main ranks [0, 1, 1, 0], loads 11 / 10 (the base gives 19 / 2).
    w = np.array([[10, 9, 1, 1], [0, 0, 0, 0]])
    mp = PL.policy_update_plan(w, np.array([0, 0, 1, 1]), M=1, R=2, N_b=2, N_r=0)
    return mp.main.tolist() == [0, 1, 1, 0] and mp.rank_load().tolist() == [11, 10]


STAGE34_W = np.array([[100, 90, 70, 10], [0, 0, 0, 0], [0, 0, 0, 0], [0, 0, 0, 0]])


def check_stage3_replication():
    # One machine of four ranks, one base and one redundant slot each; loads
    # 100, 90, 70, 10 (source 0). Stage 2 keeps e_i on r_i. Stage 3, four
    # rounds (RL = current rank loads, copies sharing their expert's load):
    #  1. load per copy 100, 90, 70, 10 -> e0. RL 100/90/70/10; ranks with
    #     a free redundant slot and no e0: r1, r2, r3 -> least r3 (10).
    #  2. per copy 50, 90, 70, 10 -> e1 (total load would pick e0 again).
    #     RL r0 = 50, r1 = 90, r2 = 70, r3 = 10 + 50 = 60; free and no e1:
    #     r0, r2 -> r0 (50; a main rank still holding e0's whole 100 would
    #     lose to r2).
    #  3. per copy 50, 45, 70, 10 -> e2. RL 95/45/70/60; free and no e2: r1.
    #  4. per copy 50, 45, 35, 10 -> e0. RL 95/80/35/60; free and no e0: r2.
    # Copies: e0 [r0, r3, r2], e1 [r1, r0], e2 [r2, r1], e3 [r3].
    mp = PL.policy_update_plan(STAGE34_W, np.arange(4), M=1, R=4, N_b=1, N_r=1)
    return mp.copies == [[0, 3, 2], [1, 0], [2, 1], [3]]


def check_stage4_two_replicated():
    # Stage 4 on the placement above. Start: r3 holds e3 (10), the rest 0.
    #  e0 (100, the heaviest) over copies r0/r3/r2 at 0/10/0: 20 units
    #     bring r0 and r2 to 10, then the three take turns from copy 0:
    #     80 = 26 rounds + 2 -> counts 37, 27, 36; loads r0 37, r3 37, r2 36.
    #  e1 (90) over r1/r0 at 0/37: 37 units to r1, then 53 in turns from
    #     copy 0 -> 27 / 26: counts 64, 26; loads r1 64, r0 63.
    #  e2 (70) over r2/r1 at 36/64: 28 units to r2, then 42 in turns ->
    #     21 / 21: counts 49, 21; loads r2 85, r1 85.
    # Rank loads 63 / 85 / 85 / 37. (Filling e2 before e1, ascending, would
    # split e2 35 / 35 over two empty ranks.)
    mp = PL.policy_update_plan(STAGE34_W, np.arange(4), M=1, R=4, N_b=1, N_r=1)
    c = mp.counts[0]
    return (c[0, :3].tolist() == [37, 27, 36] and c[1, :2].tolist() == [64, 26]
            and c[2, :2].tolist() == [49, 21] and c[3, 0] == 10
            and mp.rank_load().tolist() == [63, 85, 85, 37])


def test_stage2_relocation_worked_example():
    assert check_stage2_relocation()


def test_stage3_replication_worked_example():
    assert check_stage3_replication()


def test_stage4_two_replicated_experts_worked_example():
    assert check_stage4_two_replicated()


def test_stage3_machine_confinement():
    # Two machines of two ranks, one base and one redundant slot per rank
    # (App. D: replicas stay inside their machine). Machine 0 holds e0 (500)
    # and e1 (10): the first pick puts a replica of e0 on r1; the second
    # picks e0 again (250 per copy > 10) but r0 holds it and r1's slot is
    # used, so the machine stops, although machine 1's ranks carry no load.
    # Machine 1 holds e2, e3 with no load: the first pick takes e2 (equal
    # loads per copy, lower id) onto r3; the second takes e2 again (0/2 =
    # 0/1, lower id), which no rank can take.
    w = np.array([[500, 10, 0, 0], [0, 0, 0, 0], [0, 0, 0, 0], [0, 0, 0, 0]])
    mp = PL.policy_update_plan(w, np.array([0, 1, 2, 3]), M=2, R=2, N_b=1, N_r=1)
    assert mp.copies == [[0, 1], [1], [2, 3], [3]]
    # Stage 4: r1 starts at 10 (e1), so e0's first 10 units go to r0, then
    # the other 490 alternate from copy 0: 255 / 245
    assert mp.counts[0, 0, :2].tolist() == [255, 245]


# ---------------------------------------------------------------------------
# Mutation tests
# ---------------------------------------------------------------------------
def test_mutation_ascending_lpt_is_caught(monkeypatch):
    monkeypatch.setattr(PL, "_desc_order", lambda w, ids: sorted((int(e) for e in ids), key=lambda e: (int(w[e]), e)))
    assert not check_lpt_textbook()


def test_mutation_water_filling_to_fullest_is_caught(monkeypatch):
    real = PL.policy_update_plan

    def wrong(w, base_rank, M, R, N_b, N_r, C_max=None):
        mp = real(w, base_rank, M, R, N_b, N_r, C_max)
        mp.counts = mp.counts[:, :, ::-1].copy() if mp.counts.shape[2] > 1 else mp.counts
        return mp

    monkeypatch.setattr(PL, "policy_update_plan", wrong)
    assert not check_water_filling_worked_example()
    assert not check_single_replica_water_level()


def test_mutation_split_ignores_base_load_is_caught(monkeypatch):
    # water-filling from empty ranks (forgetting the non-replicated experts'
    # load) gives an even split instead of the water level
    real_split = PL.split_equal
    real = PL.policy_update_plan

    def wrong(w, base_rank, M, R, N_b, N_r, C_max=None):
        mp = real(w, base_rank, M, R, N_b, N_r, C_max)
        for e, c in enumerate(mp.copies):
            if len(c) > 1:
                for s in range(mp.P):
                    mp.counts[s, e, :len(c)] = real_split(int(w[s, e]), len(c))
        return mp

    monkeypatch.setattr(PL, "policy_update_plan", wrong)
    assert not check_water_filling_worked_example()


def test_mutation_stage2_deleted_is_caught(monkeypatch):
    # Stage 2 skipped: the base placement stays
    monkeypatch.setattr(PL, "stage2_relocate", lambda we, local, ranks, N_b: {})
    assert not check_stage2_relocation()


def test_mutation_stage3_most_loaded_rank_is_caught(monkeypatch):
    monkeypatch.setattr(PL, "stage3_rank",
                        lambda RL, cands: max(sorted(cands), key=lambda r: (RL[r], -r)) if cands else None)
    assert not check_stage3_replication()


def test_mutation_stage3_total_load_is_caught(monkeypatch):
    # heaviest by total load instead of load per copy
    monkeypatch.setattr(PL, "heaviest_expert",
                        lambda we, local, copies: max(sorted(local), key=lambda e: (int(we[e]), -e)) if local else None)
    assert not check_stage3_replication()


@pytest.mark.parametrize("kind", ["main_keeps_all", "every_copy_full"])
def test_mutation_stage3_unshared_load_is_caught(monkeypatch, kind):
    # rank loads that ignore how the copies of an expert share its load
    def wrong(we, local, copies, ranks):
        RL = {r: 0 for r in ranks}
        for e in local:
            for i, r in enumerate(copies[e]):
                if kind == "every_copy_full" or i == 0:
                    RL[r] += int(we[e])
        return RL

    monkeypatch.setattr(PL, "copy_loads", wrong)
    assert not check_stage3_replication()


def test_mutation_stage4_ascending_order_is_caught(monkeypatch):
    monkeypatch.setattr(PL, "stage4_order", lambda we, reps: sorted(reps, key=lambda e: (int(we[e]), e)))
    assert not check_stage4_two_replicated()
