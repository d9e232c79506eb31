"""Plain CPU oracle of ForeMoE's placement planner (Sec. 8, Alg. 1; App. D, Alg. 3).

TEST INFRASTRUCTURE. Only tests/, the smoke check and the benchmark's CPU
baseline may import or run this module; the product path never does.

It follows the paper's steps in the paper's order, one loop per step, with
exact integer arithmetic so that every decision (argmin, sort order) is
reproducible:

* Stage 1, base placement (Alg. 1): experts in descending aggregate load;
  machine-level greedy on score = c_load*(ML[m] + w_e) + c_traffic*(MC[m] +
  Delta_{m,e}); then rank-level LPT inside each machine.
* Policy-update Stages 2-4 (Alg. 3), per micro-step and per machine:
  Stage 2 LPT relocation of the machine's experts over its ranks by this
  micro-step's load; Stage 3 one replica at a time of the locally heaviest
  expert onto the least-loaded rank; Stage 4 water-filling: every token unit
  of a replicated expert goes to the copy whose rank has the least load so
  far.

Readings where the paper is silent (listed in the design notes as well):
* every sort is by descending load, ties by ascending expert id; every
  argmin over ranks takes the lowest rank id among equals, over copies the
  lowest copy index;
* a rank holds at most N_b base experts (Stage 1 and 2 skip full ranks and
  machines) and at most N_r replicas (Stage 3); a replica never goes to a
  rank that already holds a copy of the same expert; Stage 3 stops early
  when no rank can take the chosen expert;
* the time-model weights of the Stage 1 score are non-negative integers
  (the ratio n1*K1 : n2*K2), so scores are exact;
* "locally heaviest" in Stage 3 compares the load per copy w_e / c_e
  (c_e = copies so far) exactly, as w_e * c_f against w_f * c_e; after a
  replica is added, the copies of an expert share its load by the
  contiguous integer split floor(w*(i+1)/c) - floor(w*i/c) (copy 0 first),
  which is what RL holds for replicated experts during Stage 3;
* Stage 4 starts from the loads of the non-replicated experts, handles the
  replicated experts in descending load, and within an expert the source
  ranks in ascending order; copy 0 is the Stage 2 (main) placement, copies
  1.. the replicas in the order Stage 3 placed them.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional

import numpy as np


def _desc_order(w: np.ndarray, ids) -> List[int]:
    """ids sorted by descending w, ties by ascending id."""
    return sorted((int(e) for e in ids), key=lambda e: (-int(w[e]), e))


def rank_lpt(w: np.ndarray, experts, ranks: List[int], cap: int) -> dict:
    """Rank-level LPT (Alg. 1, rank-level placement; Alg. 3 Stage 2).

    Experts in descending load, each onto the least-loaded rank that still
    has a free slot (at most ``cap`` experts per rank). Returns {e: rank}.
    """
    load = {r: 0 for r in ranks}
    used = {r: 0 for r in ranks}
    out = {}
    for e in _desc_order(w, experts):
        best = None
        for r in ranks:
            if used[r] >= cap:
                continue
            if best is None or load[r] < load[best]:
                best = r
        if best is None:
            raise ValueError("not enough base slots for the experts")
        out[e] = best
        load[best] += int(w[e])
        used[best] += 1
    return out


def base_placement(w_agg: np.ndarray, M: int, R: int, N_b: int, c_load: int = 1,
                   c_traffic: int = 0) -> np.ndarray:
    """Stage 1 (Alg. 1): rank of every expert from the aggregate load.

    w_agg int [P, E] (P = M*R source ranks; source s sits on machine s // R).
    Returns int64 [E] rank ids.
    """
    w_agg = np.asarray(w_agg, dtype=np.int64)
    P, E = w_agg.shape
    if P != M * R or E > P * N_b:
        raise ValueError("shape does not fit M*R ranks with N_b base slots")
    we = w_agg.sum(axis=0)
    ML = [0] * M
    MC = [0] * M
    count = [0] * M
    machine = {}
    for e in _desc_order(we, range(E)):
        best, best_score, best_delta = None, None, None
        for m in range(M):
            if count[m] >= R * N_b:
                continue
            delta = int(sum(int(w_agg[s, e]) for s in range(P) if s // R != m))
            score = c_load * (ML[m] + int(we[e])) + c_traffic * (MC[m] + delta)
            if best is None or score < best_score:
                best, best_score, best_delta = m, score, delta
        machine[e] = best
        ML[best] += int(we[e])
        MC[best] += best_delta
        count[best] += 1
    rank = np.full(E, -1, dtype=np.int64)
    for m in range(M):
        local = [e for e in range(E) if machine[e] == m]
        for e, r in rank_lpt(we, local, list(range(m * R, (m + 1) * R)), N_b).items():
            rank[e] = r
    return rank


def split_equal(w: int, c: int) -> List[int]:
    """Contiguous integer split of w units over c copies, copy 0 first."""
    return [(w * (i + 1)) // c - (w * i) // c for i in range(c)]


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
    """Alg. 3: Stages 2-4 for one micro-step. w int [P, E] is w_{s,e}."""
    w = np.asarray(w, dtype=np.int64)
    P, E = w.shape
    we = w.sum(axis=0)
    main = np.asarray(base_rank, dtype=np.int64).copy()
    copies: List[List[int]] = [[] for _ in range(E)]
    for m in range(M):
        ranks = list(range(m * R, (m + 1) * R))
        local = [e for e in range(E) if main[e] // R == m]
        # Stage 2: LPT relocation by this micro-step's load
        for e, r in rank_lpt(we, local, ranks, N_b).items():
            main[e] = r
        for e in local:
            copies[e] = [int(main[e])]
        # Stage 3: R * N_r replicas, one at a time
        used = {r: 0 for r in ranks}

        def rank_loads():
            RL = {r: 0 for r in ranks}
            for e in local:
                for r, part in zip(copies[e], split_equal(int(we[e]), len(copies[e]))):
                    RL[r] += part
            return RL

        for _ in range(R * N_r):
            heavy = None
            for e in sorted(local):
                if heavy is None or int(we[e]) * len(copies[heavy]) > int(we[heavy]) * len(copies[e]):
                    heavy = e
            if heavy is None:
                break
            RL = rank_loads()
            best = None
            for r in ranks:
                if used[r] >= N_r or r in copies[heavy]:
                    continue
                if best is None or RL[r] < RL[best]:
                    best = r
            if best is None:
                break
            copies[heavy].append(best)
            used[best] += 1
    cmax = max(len(c) for c in copies) if C_max is None else C_max
    if any(len(c) > cmax for c in copies):
        raise ValueError("C_max below the copies placed")
    counts = np.zeros((P, E, cmax), dtype=np.int64)
    # Stage 4: water-filling, per machine
    for m in range(M):
        ranks = list(range(m * R, (m + 1) * R))
        local = [e for e in range(E) if copies[e] and copies[e][0] // R == m]
        load = {r: 0 for r in ranks}
        for e in local:
            if len(copies[e]) == 1:
                counts[:, e, 0] = w[:, e]
                load[copies[e][0]] += int(we[e])
        for e in _desc_order(we, [e for e in local if len(copies[e]) > 1]):
            for s in range(P):
                for _ in range(int(w[s, e])):
                    best = 0
                    for c in range(1, len(copies[e])):
                        if load[copies[e][c]] < load[copies[e][best]]:
                            best = c
                    counts[s, e, best] += 1
                    load[copies[e][best]] += 1
    return MicroPlan(P, E, main, copies, counts)


def imbalance(loads: np.ndarray) -> float:
    """Compute imbalance ratio L_max / mean_r L_r (Sec. 7.1 time model; the
    metric of the case study, Sec. 10.4)."""
    loads = np.asarray(loads, dtype=np.float64)
    return float(loads.max() / loads.mean()) if loads.mean() > 0 else 1.0
