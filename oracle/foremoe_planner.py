"""Plain CPU oracle of ForeMoE's placement planner (Sec. 8, Alg. 1; App. D, Alg. 3).

TEST INFRASTRUCTURE. Only tests/, the smoke check and the benchmark's CPU
baseline may import or run this module; the product path never does.

One function per rule the paper states, with exact integer arithmetic (and
exact fractions where a rule compares ratios) so that every decision
(argmin, argmax, sort order) is reproducible:

* Stage 1, base placement (Sec. 8 Stage 1): experts in descending aggregate
  load; each goes to the machine whose score, the time-model weighted sum
  of the load the machine would then hold and the cross-machine tokens it
  would then receive, is lowest (``machine_scores``); then each machine's
  experts are spread over its ranks by LPT (``rank_lpt``).
* Policy-update Stages 2-4 (App. D), per micro-step and per machine:
  Stage 2 re-runs LPT on this micro-step's load (``stage2_relocate``);
  Stage 3 fills the redundant slots one at a time with a replica of the
  locally heaviest expert on the least-loaded rank (``stage3_replicate``);
  Stage 4 hands every token unit of a replicated expert to the copy whose
  rank holds the least load so far (``stage4_water_fill``).

Readings where the paper is silent (listed in the design notes as well):
* every sort is by descending load, ties by ascending expert id; every
  argmin over machines or ranks takes the lowest id among equals, over
  copies the lowest copy index;
* a rank holds at most N_b base experts (Stages 1 and 2 skip full ranks and
  machines) and at most N_r replicas (Stage 3); a replica never goes to a
  rank that already holds a copy of the same expert; Stage 3 stops early
  when no rank can take the chosen expert;
* the time-model weights of the Stage 1 score are non-negative integers
  (the ratio n1*K1 : n2*K2), so scores are exact;
* "locally heaviest" in Stage 3 is the largest load per copy w_e / c_e
  (c_e = copies so far), compared exactly; a rank's "current load" counts
  each copy of an expert with its share of the expert's load under the
  contiguous integer split floor(w*(i+1)/c) - floor(w*i/c) (copy 0 first);
* Stage 4 starts from the loads of the non-replicated experts, handles the
  replicated experts in descending load, and within an expert the source
  ranks in ascending order; copy 0 is the Stage 2 (main) placement, copies
  1.. the replicas in the order Stage 3 placed them.
"""
from __future__ import annotations

from dataclasses import dataclass
from fractions import Fraction
from typing import Dict, List, Optional

import numpy as np

_FULL = np.iinfo(np.int64).max  # score of a machine with no free base slot


def _desc_order(w: np.ndarray, ids) -> List[int]:
    """ids sorted by descending w, ties by ascending id."""
    return sorted((int(e) for e in ids), key=lambda e: (-int(w[e]), e))


def _first_argmin(values: Dict[int, int], candidates) -> Optional[int]:
    """The candidate with the smallest value, the lowest id among equals."""
    cands = sorted(candidates)
    if not cands:
        return None
    return min(cands, key=lambda r: (values[r], r))


# ---------------------------------------------------------------------------
# LPT (Sec. 8 Stage 1, rank level; App. D Stage 2)
# ---------------------------------------------------------------------------
def rank_lpt(w: np.ndarray, experts, ranks: List[int], cap: int) -> dict:
    """Longest processing time first: experts in descending load, each onto
    the rank with the least load so far among those with a free slot (at
    most ``cap`` experts per rank). Returns {e: rank}."""
    load = {r: 0 for r in ranks}
    used = {r: 0 for r in ranks}
    out = {}
    for e in _desc_order(w, experts):
        r = _first_argmin(load, [r for r in ranks if used[r] < cap])
        if r is None:
            raise ValueError("not enough base slots for the experts")
        out[e] = r
        load[r] += int(w[e])
        used[r] += 1
    return out


# ---------------------------------------------------------------------------
# Stage 1: base placement (Sec. 8 Stage 1)
# ---------------------------------------------------------------------------
def machine_scores(w_agg: np.ndarray, e: int, ML: np.ndarray, MC: np.ndarray, R: int, c_load: int,
                   c_traffic: int) -> np.ndarray:
    """Score of placing expert e on each machine m at once:
    c_load * (load on m after placing e) + c_traffic * (cross-machine
    tokens m receives after placing e), where the tokens e adds are those
    of source ranks outside m (source s sits on machine s // R)."""
    M = ML.shape[0]
    col = w_agg[:, e].astype(np.int64)
    inside = col.reshape(M, R).sum(axis=1)
    delta = col.sum() - inside
    return c_load * (ML + col.sum()) + c_traffic * (MC + delta), delta


def base_placement(w_agg: np.ndarray, M: int, R: int, N_b: int, c_load: int = 1,
                   c_traffic: int = 0) -> np.ndarray:
    """Stage 1: rank of every expert from the aggregate load.

    w_agg int [P, E] (P = M*R source ranks; source s sits on machine s // R).
    Returns int64 [E] rank ids.
    """
    w_agg = np.asarray(w_agg, dtype=np.int64)
    P, E = w_agg.shape
    if P != M * R or E > P * N_b:
        raise ValueError("shape does not fit M*R ranks with N_b base slots")
    we = w_agg.sum(axis=0)
    ML = np.zeros(M, dtype=np.int64)
    MC = np.zeros(M, dtype=np.int64)
    hosted = np.zeros(M, dtype=np.int64)
    machine = np.full(E, -1, dtype=np.int64)
    for e in _desc_order(we, range(E)):
        score, delta = machine_scores(w_agg, e, ML, MC, R, c_load, c_traffic)
        score = np.where(hosted < R * N_b, score, _FULL)
        m = int(np.argmin(score))  # first minimum: the lowest machine id among equals
        machine[e] = m
        ML[m] += we[e]
        MC[m] += delta[m]
        hosted[m] += 1
    rank = np.full(E, -1, dtype=np.int64)
    for m in range(M):
        local = np.nonzero(machine == m)[0]
        for e, r in rank_lpt(we, local, list(range(m * R, (m + 1) * R)), N_b).items():
            rank[e] = r
    return rank


# ---------------------------------------------------------------------------
# Stages 2-4 of the policy update (App. D)
# ---------------------------------------------------------------------------
def split_equal(w: int, c: int) -> List[int]:
    """Contiguous integer split of w units over c copies, copy 0 first."""
    return [(w * (i + 1)) // c - (w * i) // c for i in range(c)]


def stage2_relocate(we: np.ndarray, local: List[int], ranks: List[int], N_b: int) -> dict:
    """Stage 2: the machine's experts spread over its ranks by LPT on this
    micro-step's load. Returns {e: rank}."""
    return rank_lpt(we, local, ranks, N_b)


def copy_loads(we: np.ndarray, local: List[int], copies: Dict[int, List[int]], ranks: List[int]) -> Dict[int, int]:
    """Current load of every rank: each copy of an expert carries its share
    of the expert's load (contiguous split, copy 0 first)."""
    RL = {r: 0 for r in ranks}
    for e in local:
        for r, part in zip(copies[e], split_equal(int(we[e]), len(copies[e]))):
            RL[r] += part
    return RL


def heaviest_expert(we: np.ndarray, local: List[int], copies: Dict[int, List[int]]) -> Optional[int]:
    """The locally heaviest expert: largest load per copy, lowest id among equals."""
    if not local:
        return None
    return max(sorted(local), key=lambda e: (Fraction(int(we[e]), len(copies[e])), -e))


def stage3_rank(RL: Dict[int, int], candidates: List[int]) -> Optional[int]:
    """The rank a Stage 3 replica goes to: least current load among the
    candidates, lowest rank id among equals."""
    return _first_argmin(RL, candidates)


def stage3_replicate(we: np.ndarray, local: List[int], copies: Dict[int, List[int]], ranks: List[int],
                     N_r: int) -> None:
    """Stage 3: R * N_r times, a replica of the locally heaviest expert on the
    rank with the least current load among those with a free redundant slot
    and no copy of that expert; stops when no rank qualifies. Appends to
    ``copies`` in place."""
    used = {r: 0 for r in ranks}
    for _ in range(len(ranks) * N_r):
        e = heaviest_expert(we, local, copies)
        if e is None:
            return
        RL = copy_loads(we, local, copies, ranks)
        r = stage3_rank(RL, [r for r in ranks if used[r] < N_r and r not in copies[e]])
        if r is None:
            return
        copies[e].append(r)
        used[r] += 1


def stage4_order(we: np.ndarray, replicated: List[int]) -> List[int]:
    """Order in which Stage 4 fills the replicated experts: descending load."""
    return _desc_order(we, replicated)


def stage4_water_fill(w: np.ndarray, local: List[int], copies: Dict[int, List[int]], ranks: List[int],
                      counts: np.ndarray) -> Dict[int, int]:
    """Stage 4: tokens of non-replicated experts stay on their one copy; then
    for each replicated expert and each source rank in ascending order,
    every token unit goes to the copy whose rank holds the least
    accumulated load (lowest copy index among equals). Writes counts
    [P, E, C] in place; returns the ranks' loads."""
    P = w.shape[0]
    we = w.sum(axis=0)
    load = {r: 0 for r in ranks}
    for e in local:
        if len(copies[e]) == 1:
            counts[:, e, 0] = w[:, e]
            load[copies[e][0]] += int(we[e])
    for e in stage4_order(we, [e for e in local if len(copies[e]) > 1]):
        c = copies[e]
        for s in range(P):
            for _ in range(int(w[s, e])):
                i = min(range(len(c)), key=lambda i: (load[c[i]], i))
                counts[s, e, i] += 1
                load[c[i]] += 1
    return load


@dataclass
class MicroPlan:
    """A micro-step's placement over all ranks.

    main[e]         rank of copy 0 (the main expert)
    copies[e]       ranks of copies 0, 1, ... (copy 0 = main[e])
    counts          int64 [P, E, C_max]: tokens of source s for expert e that
                    copy c processes (the token assignment r_{s,e,j} times
                    w_{s,e}, Sec. 7.2)
    """
    P: int
    E: int
    main: np.ndarray
    copies: List[List[int]]
    counts: np.ndarray

    def rank_load(self) -> np.ndarray:
        L = np.zeros(self.P, dtype=np.int64)
        for e in range(self.E):
            for c, r in enumerate(self.copies[e]):
                L[r] += int(self.counts[:, e, c].sum())
        return L


def policy_update_plan(w: np.ndarray, base_rank: np.ndarray, M: int, R: int, N_b: int, N_r: int,
                       C_max: Optional[int] = None) -> MicroPlan:
    """App. D: Stages 2-4 for one micro-step, machine by machine.
    w int [P, E] is w_{s,e}; base_rank [E] the Stage 1 placement."""
    w = np.asarray(w, dtype=np.int64)
    P, E = w.shape
    we = w.sum(axis=0)
    main = np.asarray(base_rank, dtype=np.int64).copy()
    copies: Dict[int, List[int]] = {e: [] for e in range(E)}
    per_machine = []
    for m in range(M):
        ranks = list(range(m * R, (m + 1) * R))
        local = [e for e in range(E) if main[e] // R == m]
        for e, r in stage2_relocate(we, local, ranks, N_b).items():
            main[e] = r
        for e in local:
            copies[e] = [int(main[e])]
        stage3_replicate(we, local, copies, ranks, N_r)
        per_machine.append((local, ranks))
    cmax = max(len(c) for c in copies.values()) if C_max is None else C_max
    if any(len(c) > cmax for c in copies.values()):
        raise ValueError("C_max below the copies placed")
    counts = np.zeros((P, E, cmax), dtype=np.int64)
    for local, ranks in per_machine:
        stage4_water_fill(w, local, copies, ranks, counts)
    return MicroPlan(P, E, main, [copies[e] for e in range(E)], counts)


def imbalance(loads: np.ndarray) -> float:
    """Compute imbalance ratio L_max / mean_r L_r (Sec. 7.1 time model; the
    metric of the case study, Sec. 10.4)."""
    loads = np.asarray(loads, dtype=np.float64)
    return float(loads.max() / loads.mean()) if loads.mean() > 0 else 1.0
