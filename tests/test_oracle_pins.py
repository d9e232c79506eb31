"""Pins of the fp64 oracle against facts fixed outside the oracle itself.

Every check here is an independent formulation: brute force on tiny inputs,
invariants of the MILP constraints (Sec. 7.2, App. C), a dense non-MoE
reference of the MoE layer (Sec. 2.1), a plain SwiGLU MLP written in pure
Python (App. A), placement invariance, central finite differences of the
backward, and the analytic numbers printed in App. A.4. Mutation tests plant
plausible mistakes in the oracle (on the CPU) and require a pin to catch them.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle.foremoe_oracle as O
from workload import accounting as acc
from workload import make_custom, make_workload, plan_from_slots

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rel_err(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


# ---------------------------------------------------------------------------
# Histogram
# ---------------------------------------------------------------------------
def check_histogram_brute_force():
    rng = np.random.default_rng(0)
    E = 5
    ids = rng.integers(-3, E + 2, size=(37, 3)).astype(np.int32)
    counts, invalid = O.histogram(ids, E)
    exp = [0] * E
    inv = 0
    for v in ids.reshape(-1).tolist():
        if v == -1:
            continue
        if 0 <= v < E:
            exp[v] += 1
        else:
            inv += 1
    return counts.tolist() == exp and invalid == inv


def test_histogram_brute_force():
    assert check_histogram_brute_force()


def test_histogram_sum_equals_pairs():
    w = make_workload("tiny-fp32")
    m = w.micro[0]
    ids = m.ids.copy()
    ids[::7, 1] = -1
    counts, invalid = O.histogram(ids, w.spec.E)
    assert invalid == 0
    assert int(counts.sum()) == ids.size - int(np.count_nonzero(ids == -1))


# ---------------------------------------------------------------------------
# Replica split
# ---------------------------------------------------------------------------
def check_replica_bounds_brute_force():
    for n in range(0, 65):
        for R in range(1, 5):
            for w in itertools.product(range(0, 4), repeat=R):
                if sum(w) == 0:
                    continue
                B = O.replica_bounds(n, list(w))
                W = sum(w)
                pref = 0
                exp = [0]
                for wi in w:
                    pref += wi
                    # largest b in [0, n] with b * W <= n * pref, by enumeration
                    b = max(b for b in range(n + 1) if b * W <= n * pref)
                    exp.append(b)
                if B != exp:
                    return False
    return True


def test_replica_bounds_brute_force():
    assert check_replica_bounds_brute_force()


def test_replica_bounds_cover_and_balance():
    for n in range(0, 200):
        for R in range(1, 6):
            B = O.replica_bounds(n, [1] * R)
            assert B[0] == 0 and B[-1] == n
            sizes = [B[r + 1] - B[r] for r in range(R)]
            assert all(s >= 0 for s in sizes)
            assert max(sizes) - min(sizes) <= 1      # equal weights: balanced split
            assert sum(sizes) == n                    # token conservation


def test_assign_offsets_are_prefix_sums():
    w = make_workload("tiny-fp32")
    m = w.micro[0]
    counts, _ = O.histogram(m.ids, w.spec.E)
    rep_begin, slot_count, slot_offset = O.assign_replicas(counts, m.plan)
    assert slot_offset[0] == 0
    assert list(np.diff(slot_offset)) == list(slot_count)
    # expert 0 has two local replicas; both halves together cover its list
    assert slot_count[0] + slot_count[3] == counts[0]
    assert slot_count[0] == counts[0] // 2
    assert int(slot_offset[-1]) == int(counts[0] + counts[1] + counts[2])


# ---------------------------------------------------------------------------
# Permute
# ---------------------------------------------------------------------------
def _brute_dispatch(ids, plan):
    """Row of every pair by brute force: rank by counting, slot by scanning."""
    T, K = ids.shape
    flat = ids.reshape(-1).tolist()
    counts = [flat.count(e) for e in range(plan.E)]
    wts = None if plan.expert_rep_weight is None else np.asarray(plan.expert_rep_weight).reshape(plan.E, plan.R_max)
    slot_of = {}
    for j in range(plan.S):
        slot_of[(int(plan.slot_expert[j]), int(plan.slot_replica[j]))] = j
    pair_slot = {}
    for p, e in enumerate(flat):
        if not (0 <= e < plan.E):
            continue
        q = sum(1 for p2 in range(p) if flat[p2] == e)
        R = int(plan.expert_nrep[e])
        w = [1] * R if wts is None else [int(v) for v in wts[e, :R]]
        W = sum(w)
        pref = 0
        for r in range(R):
            lo = max(b for b in range(counts[e] + 1) if b * W <= counts[e] * pref)
            pref += w[r]
            hi = max(b for b in range(counts[e] + 1) if b * W <= counts[e] * pref)
            if lo <= q < hi:
                if (e, r) in slot_of:
                    pair_slot[p] = slot_of[(e, r)]
                break
    per_slot = [sorted(p for p, j in pair_slot.items() if j == jj) for jj in range(plan.S)]
    offsets = [0]
    for lst in per_slot:
        offsets.append(offsets[-1] + len(lst))
    pair_to_row = [-1] * (T * K)
    for j, lst in enumerate(per_slot):
        for i, p in enumerate(lst):
            pair_to_row[p] = offsets[j] + i
    return pair_to_row, offsets


def _run_dispatch(ids, x, plan, n_cap):
    counts, _ = O.histogram(ids, plan.E)
    rep_begin, slot_count, slot_offset = O.assign_replicas(counts, plan)
    x_perm, r2p, p2r, dropped = O.permute(x, ids, plan, rep_begin, slot_offset, n_cap)
    return slot_offset, x_perm, r2p, p2r, dropped


def _tiny_dispatch_case():
    rng = np.random.default_rng(3)
    T, K, E = 29, 3, 6
    ids = rng.integers(0, E, size=(T, K)).astype(np.int32)
    ids[4, 1] = -1
    x = rng.standard_normal((T, 5))
    plan = plan_from_slots(E, [(2, 0), (0, 0), (0, 2), (5, 0), (3, 1), (1, 0)],
                           nrep={0: 3, 3: 2}, rep_weights={0: [1, 0, 3], 3: [2, 1]})
    return ids, x, plan


def check_permute_brute_force():
    ids, x, plan = _tiny_dispatch_case()
    T, K = ids.shape
    slot_offset, x_perm, r2p, p2r, dropped = _run_dispatch(ids, x, plan, T * K)
    exp_p2r, exp_off = _brute_dispatch(ids, plan)
    if list(slot_offset) != exp_off or list(p2r) != exp_p2r or dropped != 0:
        return False
    for p, row in enumerate(exp_p2r):
        if row >= 0 and (r2p[row] != p or not np.array_equal(x_perm[row], x[p // K])):
            return False
    return True


def test_permute_brute_force():
    assert check_permute_brute_force()


def test_permute_invariants_tiny():
    w = make_workload("tiny-fp32")
    m = w.micro[0]
    T, K = m.ids.shape
    x = w.x(0)
    slot_offset, x_perm, r2p, p2r, dropped = _run_dispatch(m.ids, x, m.plan, T * K)
    N = int(slot_offset[-1])
    rows = r2p[:N]
    assert len(set(rows.tolist())) == N                      # injective
    assert np.all(p2r[rows] == np.arange(N))                 # inverse maps
    assert np.all(r2p[N:] == -1)
    for j in range(m.plan.S):
        seg = rows[slot_offset[j]:slot_offset[j + 1]]
        assert np.all(m.ids.reshape(-1)[seg] == m.plan.slot_expert[j])   # feasibility
        assert np.all(np.diff(seg) > 0)                      # ascending pair order
    local = np.isin(m.ids.reshape(-1), m.plan.local_experts)
    assert np.all((p2r >= 0) == local)                       # every local pair exactly once


def test_permute_overflow_drops_tail():
    ids, x, plan = _tiny_dispatch_case()
    T, K = ids.shape
    full = _run_dispatch(ids, x, plan, T * K)
    N = int(full[0][-1])
    cap = N - 5
    slot_offset, x_perm, r2p, p2r, dropped = _run_dispatch(ids, x, plan, cap)
    assert dropped == 5
    assert np.all(p2r[p2r >= 0] < cap)
    assert np.array_equal(np.where(full[3] >= cap, -1, full[3]), p2r)


def test_every_pair_dispatched_once_over_all_ranks():
    """Coverage + conservation over a whole EP group (App. C): simulate every
    rank's slot table; each valid pair lands on exactly one slot."""
    rng = np.random.default_rng(11)
    T, K, E, P = 64, 4, 16, 4
    ids = rng.integers(0, E, size=(T, K)).astype(np.int32)
    ids[rng.random((T, K)) < 0.05] = -1
    nrep = {0: 3, 5: 2, 9: 2}
    weights = {0: [2, 1, 1], 5: [1, 3], 9: [1, 1]}
    extra = {1: [(0, 1), (9, 1)], 2: [(0, 2)], 3: [(5, 1)]}
    seen = np.zeros(T * K, dtype=np.int64)
    for r in range(P):
        slots = [(e, 0) for e in range(E) if e // (E // P) == r] + extra.get(r, [])
        plan = plan_from_slots(E, slots, nrep=nrep, rep_weights=weights, R_max=3)
        _, _, r2p, p2r, _ = _run_dispatch(ids, rng.standard_normal((T, 2)), plan, T * K)
        seen[p2r >= 0] += 1
    flat = ids.reshape(-1)
    assert np.all(seen[flat >= 0] == 1)
    assert np.all(seen[flat < 0] == 0)


# ---------------------------------------------------------------------------
# FFN + combine against a dense non-MoE reference (Sec. 2.1, App. A)
# ---------------------------------------------------------------------------
def _token_ffn(xt, wgu, wd):
    F = wgu.shape[0] // 2
    a = wgu[:F] @ xt
    u = wgu[F:] @ xt
    h = a * u / (1.0 + np.exp(-a))
    return wd @ h


def dense_reference(x, ids, gates, experts, w_gate_up, w_down):
    """Every token runs every local expert; the output is masked by the gate
    mass G[t, e] = sum_k [ids[t,k] == e] * gates[t,k]."""
    T, K = ids.shape
    y = np.zeros((T, x.shape[1]))
    for t in range(T):
        for wi, e in enumerate(experts):
            G = sum(float(gates[t, k]) for k in range(K) if ids[t, k] == e)
            y[t] += G * _token_ffn(np.asarray(x[t], np.float64), np.asarray(w_gate_up[wi], np.float64),
                                   np.asarray(w_down[wi], np.float64))
    return y


def check_dense_reference():
    w = make_custom(T=40, d=16, F=24, E=6, K=2, dtype="f32", P=1, n_rep=2, seed=5)
    m = w.micro[0]
    gu, dn = w.weights(m.plan)
    x = w.x(0)
    fwd = O.layer_forward(x, m.ids, m.gates, m.plan, gu, dn)
    ref = dense_reference(x, m.ids, m.gates, list(m.plan.local_experts), gu, dn)
    return rel_err(fwd["y"], ref)


def test_dense_reference():
    assert check_dense_reference() <= 1e-12


def test_dense_reference_tiny():
    w = make_workload("tiny-fp32")
    m = w.micro[0]
    gu, dn = w.weights(m.plan)
    x = w.x(0)
    fwd = O.layer_forward(x, m.ids, m.gates, m.plan, gu, dn)
    ref = dense_reference(x, m.ids, m.gates, list(m.plan.local_experts), gu, dn)
    assert rel_err(fwd["y"], ref) <= 1e-12
    # tokens with no local pair produce zero rows
    nolocal = ~np.isin(m.ids, m.plan.local_experts).any(axis=1)
    assert nolocal.any() and np.all(fwd["y"][nolocal] == 0.0)


def check_plain_swiglu():
    """E = K = R = 1 with gate 1 is a plain SwiGLU MLP, written in pure Python."""
    rng = np.random.default_rng(2)
    T, d, F = 3, 4, 5
    x = rng.standard_normal((T, d))
    wgu = rng.standard_normal((1, 2 * F, d))
    wd = rng.standard_normal((1, d, F))
    ids = np.zeros((T, 1), dtype=np.int32)
    gates = np.ones((T, 1))
    plan = plan_from_slots(1, [(0, 0)])
    y = O.layer_forward(x, ids, gates, plan, wgu, wd)["y"]
    exp = []
    for t in range(T):
        h = []
        for f in range(F):
            a = sum(wgu[0, f, c] * x[t, c] for c in range(d))
            u = sum(wgu[0, F + f, c] * x[t, c] for c in range(d))
            h.append(a / (1.0 + math.exp(-a)) * u)
        exp.append([sum(wd[0, i, f] * h[f] for f in range(F)) for i in range(d)])
    return rel_err(y, np.array(exp))


def test_plain_swiglu_mlp():
    assert check_plain_swiglu() <= 1e-12


def test_zero_gate_is_no_contribution():
    w = make_custom(T=32, d=8, F=16, E=4, K=2, dtype="f32", P=1, n_rep=1, seed=9)
    m = w.micro[0]
    gu, dn = w.weights(m.plan)
    x = w.x(0)
    gates = m.gates.copy()
    gates[:, 1] = 0.0
    ids_drop = m.ids.copy()
    ids_drop[:, 1] = -1
    a = O.layer_forward(x, m.ids, gates, m.plan, gu, dn)["y"]
    b = O.layer_forward(x, ids_drop, gates, m.plan, gu, dn)["y"]
    assert rel_err(a, b) <= 1e-12


# ---------------------------------------------------------------------------
# Placement invariance (replication changes where, never what)
# ---------------------------------------------------------------------------
def test_placement_invariance():
    w = make_custom(T=48, d=8, F=12, E=5, K=2, dtype="f32", P=1, n_rep=0, seed=13)
    m = w.micro[0]
    T, K = m.ids.shape
    x = w.x(0)
    rng = np.random.default_rng(1)
    dy = rng.standard_normal((T, 8))
    E = 5
    plan_a = plan_from_slots(E, [(e, 0) for e in range(E)])
    plan_b = plan_from_slots(E, [(3, 1), (0, 0), (3, 0), (1, 0), (3, 2), (2, 0), (4, 0), (1, 1)],
                             nrep={3: 3, 1: 2}, rep_weights={3: [1, 2, 3], 1: [5, 1]})
    outs = []
    for plan in (plan_a, plan_b):
        gu = np.stack([w.expert_weights(int(e))[0] for e in plan.local_experts])
        dn = np.stack([w.expert_weights(int(e))[1] for e in plan.local_experts])
        fwd = O.layer_forward(x, m.ids, m.gates, plan, gu, dn)
        bwd = O.layer_backward(fwd, dy, m.gates, plan, gu, dn, T, K)
        order = np.argsort(plan.local_experts)
        outs.append((fwd["y"], bwd["dx"], bwd["dgates"], bwd["dw_gate_up"][order], bwd["dw_down"][order]))
    for a, b in zip(*outs):
        assert rel_err(a, b) <= 1e-12


# ---------------------------------------------------------------------------
# Backward by central finite differences
# ---------------------------------------------------------------------------
def check_finite_differences():
    rng = np.random.default_rng(21)
    T, d, F, E, K = 16, 8, 12, 4, 2
    ids = np.stack([rng.choice(E, size=K, replace=False) for _ in range(T)]).astype(np.int32)
    gates = rng.random((T, K))
    gates /= gates.sum(axis=1, keepdims=True)
    plan = plan_from_slots(E, [(0, 0), (1, 0), (2, 0), (3, 0), (1, 1), (3, 1)],
                           rep_weights={1: [1, 2], 3: [1, 1]})
    gu = rng.standard_normal((E, 2 * F, d)) / np.sqrt(d)
    dn = rng.standard_normal((E, d, F)) / np.sqrt(F)
    order = [int(e) for e in plan.local_experts]
    gu = gu[order]
    dn = dn[order]
    x = rng.standard_normal((T, d))
    dy = rng.standard_normal((T, d))

    def loss(x_, g_, gu_, dn_):
        return float(np.sum(dy * O.layer_forward(x_, ids, g_, plan, gu_, dn_)["y"]))

    fwd = O.layer_forward(x, ids, gates, plan, gu, dn)
    bwd = O.layer_backward(fwd, dy, gates, plan, gu, dn, T, K)
    eps = 1e-6
    worst = 0.0

    def fd(arr, idx, fn):
        old = arr[idx]
        arr[idx] = old + eps
        lp = fn()
        arr[idx] = old - eps
        lm = fn()
        arr[idx] = old
        return (lp - lm) / (2 * eps)

    for idx in [(0, 0), (3, 5), (15, 7), (8, 2)]:
        num = fd(x, idx, lambda: loss(x, gates, gu, dn))
        worst = max(worst, abs(num - bwd["dx"][idx]) / max(abs(num), 1e-3))
    for idx in [(0, 0), (5, 1), (15, 1)]:
        num = fd(gates, idx, lambda: loss(x, gates, gu, dn))
        worst = max(worst, abs(num - bwd["dgates"][idx]) / max(abs(num), 1e-3))
    for idx in [(1, 3, 4), (1, F + 2, 7), (3, 0, 0), (0, 2 * F - 1, 1)]:
        num = fd(gu, idx, lambda: loss(x, gates, gu, dn))
        worst = max(worst, abs(num - bwd["dw_gate_up"][idx]) / max(abs(num), 1e-3))
    for idx in [(1, 2, 5), (3, 7, 11), (0, 0, 0)]:
        num = fd(dn, idx, lambda: loss(x, gates, gu, dn))
        worst = max(worst, abs(num - bwd["dw_down"][idx]) / max(abs(num), 1e-3))
    return worst


def test_backward_finite_differences():
    assert check_finite_differences() <= 1e-6


def test_wgrad_accumulates_over_micro_steps():
    w = make_custom(T=24, d=8, F=8, E=3, K=2, dtype="f32", P=1, n_rep=1, micro_steps=2, seed=4)
    rng = np.random.default_rng(0)
    acc_gu = acc_dn = None
    singles = []
    for m in w.micro:
        plan = m.plan
        gu = np.stack([w.expert_weights(int(e))[0] for e in plan.local_experts])
        dn = np.stack([w.expert_weights(int(e))[1] for e in plan.local_experts])
        dy = rng.standard_normal((24, 8))
        fwd = O.layer_forward(w.x(m.index), m.ids, m.gates, plan, gu, dn)
        one = O.layer_backward(fwd, dy, m.gates, plan, gu, dn, 24, 2)
        order = np.argsort(plan.local_experts)
        singles.append((one["dw_gate_up"][order], one["dw_down"][order]))
        if acc_gu is None:
            acc_gu = np.zeros_like(one["dw_gate_up"])
            acc_dn = np.zeros_like(one["dw_down"])
        O.layer_backward(fwd, dy, m.gates, plan, gu, dn, 24, 2, acc_gu, acc_dn)
    assert rel_err(acc_gu, singles[0][0] + singles[1][0]) <= 1e-12
    assert rel_err(acc_dn, singles[0][1] + singles[1][1]) <= 1e-12


# ---------------------------------------------------------------------------
# App. A.4 printed numbers pin the FLOP and byte formulas used for rooflines
# ---------------------------------------------------------------------------
def test_appendix_a_instantiation():
    with open(os.path.join(GOLDEN, "appendix_a_qwen3_h20.json")) as f:
        g = json.load(f)
    i, p = g["inputs"], g["printed"]
    MiB, GiB = 2.0 ** 20, 2.0 ** 30
    S_e = acc.expert_bytes(i["h"], i["h_ff"], i["p_w"])
    S_g = acc.expert_bytes(i["h"], i["h_ff"], i["p_g"])
    assert S_e / MiB == p["S_e_MiB"] and S_g / MiB == p["S_g_MiB"]
    assert i["L"] * i["E"] * S_e / GiB == p["host_params_GiB_per_worker"]
    assert i["L"] * i["E"] * S_g / GiB == p["host_grads_GiB_per_worker"]
    ncpu = acc.n_min_cpu(i["h"], i["h_ff"], i["K"], i["E"], i["N_s"], i["p_w"], i["F_flops"], i["B_pcie"])
    nnv = acc.n_min_nvlink(i["h"], i["h_ff"], i["N_s"], i["p_w"], i["p_g"], i["F_flops"], i["B_nvlink"])
    assert math.floor(ncpu) == p["n_min_cpu_tokens"]
    assert math.floor(nnv) == p["n_min_nvlink_tokens"]
    n = i["n"]
    t_attn = acc.attn_flops(n, i["h"]) / i["F_flops"] * 1e3
    t_moe = acc.moe_flops(n, i["h"], i["h_ff"], i["K"], i["E"]) / i["F_flops"] * 1e3
    assert round(t_attn, 1) == p["T_attn_ms"]
    assert round(t_attn + t_moe, 1) == p["T_layer_ms"]
    # the expert-FFN term of Eq. flops_moe is 6 K n h h_ff
    assert acc.ffn_fwd_flops(i["K"] * n, i["h"], i["h_ff"]) == 6 * i["K"] * n * i["h"] * i["h_ff"]
    pre = i["N_s"] * S_e
    swap = i["N_s"] * (S_e + S_g)
    assert pre / MiB == p["prefetch_MiB"] and swap / MiB == p["swap_MiB"]
    assert round(pre / i["B_pcie"] * 1e3, 2) == p["prefetch_ms"]
    assert round(swap / i["B_nvlink"] * 1e3, 2) == p["swap_ms"]
    assert round(t_attn / (swap / i["B_nvlink"] * 1e3), 1) == p["swap_margin"]


# ---------------------------------------------------------------------------
# Mutation tests: plausible mistakes planted in the oracle must be caught
# ---------------------------------------------------------------------------
def test_mutation_silu_without_sigmoid_is_caught(monkeypatch):
    monkeypatch.setattr(O, "silu", lambda a: a)
    assert check_plain_swiglu() > 1e-3


def test_mutation_ceil_split_is_caught(monkeypatch):
    real = O.replica_bounds

    def ceil_bounds(n, weights):
        total = sum(weights)
        out, pref = [0], 0
        for w in weights:
            pref += w
            out.append(-((-n * pref) // total))
        return out

    monkeypatch.setattr(O, "replica_bounds", ceil_bounds)
    assert not check_replica_bounds_brute_force()
    assert not check_permute_brute_force()
    monkeypatch.setattr(O, "replica_bounds", real)


def test_mutation_transposed_down_is_caught(monkeypatch):
    real = O.ffn_forward

    def wrong(x_perm, slot_offset, slot_widx, w_gate_up, w_down):
        F = w_gate_up.shape[1] // 2
        # swap gate and up halves: a transposed operand layout
        swapped = np.concatenate([w_gate_up[:, F:], w_gate_up[:, :F]], axis=1)
        return real(x_perm, slot_offset, slot_widx, swapped, w_down)

    monkeypatch.setattr(O, "ffn_forward", wrong)
    assert check_dense_reference() > 1e-3


def test_mutation_dgrad_sign_is_caught(monkeypatch):
    real = O.ffn_dgrad

    def wrong(*args, **kw):
        out = real(*args, **kw)
        out["dA"] = -out["dA"]
        return out

    monkeypatch.setattr(O, "ffn_dgrad", wrong)
    assert check_finite_differences() > 1e-3


def test_mutation_combine_index_is_caught(monkeypatch):
    real = O.combine

    def wrong(y_perm, pair_to_row, gates, T, K):
        g = np.asarray(gates).reshape(T, K)[:, ::-1]   # gate of the wrong k
        return real(y_perm, pair_to_row, g, T, K)

    monkeypatch.setattr(O, "combine", wrong)
    assert check_dense_reference() > 1e-3


def test_mutation_unstable_rank_is_caught(monkeypatch):
    real = O.permute

    def wrong(x, ids, plan, rep_begin, slot_offset, n_cap):
        xp, r2p, p2r, dr = real(x, ids, plan, rep_begin, slot_offset, n_cap)
        # reverse the order within each slot (a non-canonical ranking)
        for j in range(plan.S):
            lo, hi = int(slot_offset[j]), int(slot_offset[j + 1])
            r2p[lo:hi] = r2p[lo:hi][::-1].copy()
            xp[lo:hi] = xp[lo:hi][::-1].copy()
        for row in range(int(slot_offset[-1])):
            p2r[r2p[row]] = row
        return xp, r2p, p2r, dr

    monkeypatch.setattr(O, "permute", wrong)
    assert not check_permute_brute_force()
