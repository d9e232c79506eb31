"""Pins of the oracle's per-source replica split (Sec. 7.2: the token
assignment r_{s,e,j} is a fraction per source rank s; App. D Stage 4).

Independent checks: a hand-worked dispatch, reduction to the single-source
oracle (itself pinned by brute force), the floor bound and conservation of
every (source, expert) block, exact reproduction of planner counts used as
weights, and ascending pair order inside every slot. A mutation test plants
a source-blind split and requires a pin to catch it.
"""
import dataclasses

import numpy as np
import pytest

import oracle.foremoe_oracle as O
from workload import make_workload, plan_from_slots


def with_sources(plan, tb, w=None):
    return dataclasses.replace(plan, src_token_begin=np.asarray(tb, dtype=np.int32),
                               src_rep_weight=None if w is None else np.asarray(w, dtype=np.int32))


def dispatch(ids, plan, E, tb, d=2):
    T, K = ids.shape
    x = np.arange(T * d, dtype=np.float64).reshape(T, d)
    cs = O.histogram_src(ids, E, tb)
    rb, sc, so = O.assign_replicas_src(cs, plan)
    xp, r2p, p2r, dropped = O.permute_src(x, ids, plan, rb, so, T * K, tb)
    return cs, rb, sc, so, r2p, p2r


def check_hand_worked():
    # 4 tokens, top-1, one expert with two local replicas; source 0 owns
    # tokens 0-1 and splits its 2 pairs 1:1, source 1 owns tokens 2-3 and
    # sends both pairs to replica 1. Blocks: B[0] = (0, 1, 2), B[1] = (0, 0, 2).
    # Slot 0 (replica 0): p0. Slot 1 (replica 1): p1 (source 0), p2, p3.
    ids = np.zeros((4, 1), dtype=np.int32)
    plan = with_sources(plan_from_slots(1, [(0, 0), (0, 1)], R_max=2), [0, 2, 4], [[[1, 1]], [[0, 2]]])
    cs, rb, sc, so, r2p, p2r = dispatch(ids, plan, 1, [0, 2, 4])
    return (cs.tolist() == [[2], [2]] and rb.tolist() == [[[0, 1, 2]], [[0, 0, 2]]] and sc.tolist() == [1, 3]
            and so.tolist() == [0, 1, 4] and r2p[:4].tolist() == [0, 1, 2, 3] and p2r.tolist() == [0, 1, 2, 3])


def test_hand_worked():
    assert check_hand_worked()


def test_single_source_reduces_to_the_plain_split():
    w = make_workload("tiny-fp32")
    m = w.micro[0]
    T, K = m.ids.shape
    tb = [0, T]
    plan = with_sources(m.plan, tb)
    x = np.random.default_rng(0).standard_normal((T, 4))
    cs = O.histogram_src(m.ids, w.spec.E, tb)
    counts, _ = O.histogram(m.ids, w.spec.E)
    assert cs[0].tolist() == counts.tolist()
    rb_s, sc_s, so_s = O.assign_replicas_src(cs, plan)
    rb, sc, so = O.assign_replicas(counts, m.plan)
    assert np.array_equal(rb_s[0], rb) and np.array_equal(sc_s, sc) and np.array_equal(so_s, so)
    a = O.permute_src(x, m.ids, plan, rb_s, so_s, T * K, tb)
    b = O.permute(x, m.ids, m.plan, rb, so, T * K)
    assert all(np.array_equal(u, v) for u, v in zip(a[:3], b[:3])) and a[3] == b[3]


def random_case(seed, n_src=4, T=96, K=3, E=6):
    rng = np.random.default_rng(seed)
    ids = rng.integers(-1, E, size=(T, K)).astype(np.int32)
    slots = [(e, 0) for e in range(E)] + [(0, 1), (0, 2), (3, 1)]
    plan = plan_from_slots(E, slots, R_max=3)
    cuts = np.sort(rng.integers(0, T + 1, size=n_src - 1))
    tb = np.concatenate([[0], cuts, [T]]).astype(np.int32)
    wts = rng.integers(0, 4, size=(n_src, E, 3)).astype(np.int32)
    wts[:, :, 0] += 1  # positive sums
    return ids, with_sources(plan, tb, wts), tb


@pytest.mark.parametrize("seed", range(5))
def test_floor_bound_conservation_and_order(seed):
    ids, plan, tb = random_case(seed)
    E = plan.E
    cs, rb, sc, so, r2p, p2r = dispatch(ids, plan, E, tb)
    n_src = len(tb) - 1
    for s in range(n_src):
        for e in range(E):
            R = int(plan.expert_nrep[e])
            cnt = np.diff(rb[s, e, :R + 1])
            n = int(cs[s, e])
            wt = plan.src_rep_weight[s, e, :R].astype(np.float64)
            assert cnt.sum() == n and (cnt >= 0).all()
            assert np.all(np.abs(cnt - n * wt / wt.sum()) < 1.0)
    # every pair of an expert with all replicas local lands exactly once,
    # inside a slot of its expert; rows of a slot in ascending p
    flat = ids.reshape(-1)
    for p, e in enumerate(flat.tolist()):
        if e < 0:
            continue
        row = p2r[p]
        assert row >= 0 and r2p[row] == p
        j = int(np.searchsorted(so, row, side="right") - 1)
        assert plan.slot_expert[j] == e
    for j in range(plan.S):
        rows = r2p[so[j]:so[j + 1]]
        assert (np.diff(rows) > 0).all()


def test_planner_counts_as_weights_are_reproduced():
    # weights equal to exact per-(source, expert, copy) token counts (what
    # the planner's water-filling produces) give exactly those blocks
    ids, plan, tb = random_case(11)
    cs = O.histogram_src(ids, plan.E, tb)
    rng = np.random.default_rng(3)
    exact = np.zeros_like(plan.src_rep_weight)
    for s in range(len(tb) - 1):
        for e in range(plan.E):
            R = int(plan.expert_nrep[e])
            cut = np.sort(rng.integers(0, cs[s, e] + 1, size=R - 1))
            exact[s, e, :R] = np.diff(np.concatenate([[0], cut, [cs[s, e]]]))
    plan = dataclasses.replace(plan, src_rep_weight=exact)
    rb, _, _ = O.assign_replicas_src(cs, plan)
    for s in range(len(tb) - 1):
        for e in range(plan.E):
            R = int(plan.expert_nrep[e])
            assert np.diff(rb[s, e, :R + 1]).tolist() == exact[s, e, :R].tolist()


def test_mutation_source_blind_split_is_caught(monkeypatch):
    # splitting each expert's global list with the first source's weights
    # (ignoring where the tokens come from) must be caught
    real = O.assign_replicas_src

    def wrong(counts_src, plan):
        tot = np.asarray(counts_src).sum(axis=0, keepdims=True)
        rb, sc, so = real(tot, dataclasses.replace(plan, src_rep_weight=np.asarray(plan.src_rep_weight)[:1]))
        return np.repeat(rb, np.asarray(counts_src).shape[0], axis=0), sc, so

    monkeypatch.setattr(O, "assign_replicas_src", wrong)
    assert not check_hand_worked()
