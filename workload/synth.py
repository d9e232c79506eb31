"""Seeded synthetic micro-step workloads shaped like the paper's RL routing.

The paper measures on rollout routing recorded from Qwen3 models on the
DAPO-Math-17k and CodeForces datasets (Sec. 10, setup). Neither the weights
nor the datasets are available, so this module stands in for them with a
recipe that reproduces the two load properties the paper reports (Sec. 3,
"Step-level: stable but skewed" and "Micro-step-level: highly variable and
skewed"):

* step-level popularity is a fixed Zipf law over experts, z_e = (pi(e)+1)^-s;
* each micro-step multiplies it by a mean-one Dirichlet(alpha) factor,
  bias_e = ln z_e + ln max(E * g_e, 1e-30), g ~ Dirichlet(alpha * 1_E);
* router logits are N(0,1) + bias_e; the recorded top-K ids are the K
  largest logits (descending, ties to the lower id) and the gates are the
  softmax probabilities of those experts renormalised over the K picks
  (Sec. 2.1: router probabilities weight the selected experts).

The placement plan stands in for the paper's planner (Sec. 7):

* a base placement by rank-level LPT (Alg. 1 with a single machine) over the
  aggregate load of all generated micro-steps, with the capacity of E/P base
  slots per rank enforced (least-loaded rank with a free base slot, ties to
  the lower rank id);
* the measured rank is the one whose aggregate load is closest to the mean;
* per micro-step, the rank's N_r locally heaviest hosted experts get one
  replica each in a redundant slot (Alg. 3, Stage 3), both replicas local,
  with an equal token split.

Nothing here computes any part of the expert layer itself. Random numbers
come from numpy's PCG64 keyed by SeedSequence(seed, spawn_key=...), so every
array is reproducible on any host. Floating-point values are drawn in
float32 and, for bf16 workloads, rounded to bfloat16 (ties to even).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from .bf16 import bf16_round


@dataclass(frozen=True)
class ConfigSpec:
    cid: int
    name: str
    T: int              # tokens per micro-step
    d: int              # model width (paper: h)
    F: int              # expert FFN width (paper: h_ff)
    E: int              # experts
    K: int              # top-k
    dtype: str          # "f32" or "bf16"
    zipf_s: float
    alpha: Optional[float]  # Dirichlet jitter; None = no micro-step jitter
    permute_popularity: bool
    P: int              # EP ranks the base placement is planned over
    n_rep: int          # redundant slots on the measured rank (paper: N_r)
    micro_steps: int    # micro-steps generated (for planning and the policy update)
    backward: bool
    seed: int


CONFIGS: Dict[int, ConfigSpec] = {
    1: ConfigSpec(1, "tiny-fp32", T=256, d=128, F=256, E=8, K=2, dtype="f32",
                  zipf_s=1.2, alpha=None, permute_popularity=False, P=1, n_rep=1,
                  micro_steps=1, backward=True, seed=1001),
    2: ConfigSpec(2, "mixtral-8x7b-share", T=4096, d=4096, F=14336, E=8, K=2, dtype="bf16",
                  zipf_s=1.0, alpha=0.5, permute_popularity=False, P=1, n_rep=2,
                  micro_steps=1, backward=False, seed=1002),
    3: ConfigSpec(3, "qwen3-30b-a3b-ep8-share", T=16384, d=2048, F=768, E=128, K=8, dtype="bf16",
                  zipf_s=1.1, alpha=0.3, permute_popularity=True, P=8, n_rep=4,
                  micro_steps=16, backward=False, seed=1003),
    4: ConfigSpec(4, "deepseek-v3-ep32-share", T=32768, d=7168, F=2048, E=256, K=8, dtype="bf16",
                  zipf_s=1.3, alpha=0.2, permute_popularity=True, P=32, n_rep=2,
                  micro_steps=16, backward=False, seed=1004),
    # The policy-update stage runs on the same share and micro-steps as config 3.
    5: ConfigSpec(5, "qwen3-30b-a3b-ep8-policy-update", T=16384, d=2048, F=768, E=128, K=8,
                  dtype="bf16", zipf_s=1.1, alpha=0.3, permute_popularity=True, P=8, n_rep=4,
                  micro_steps=16, backward=True, seed=1003),
}

# workload id by name
CONFIG_IDS: Dict[str, int] = {spec.name: i for i, spec in CONFIGS.items()}


@dataclass
class Plan:
    """One micro-step's slot table for the local GPU (paper Sec. 7 terminology).

    Slot j holds replica ``slot_replica[j]`` of expert ``slot_expert[j]``.
    Expert e has ``expert_nrep[e]`` replicas in the whole EP group (local or
    not); its token list is split among them by the integer weights
    ``expert_rep_weight[e, :R_e]`` (None = equal). ``slot_widx`` selects the
    weight matrices a slot computes with and ``slot_gidx`` the main-expert
    gradient it accumulates into; ``local_experts[w]`` is the global expert id
    of weight/gradient index w.
    """
    E: int
    R_max: int
    slot_expert: np.ndarray
    slot_replica: np.ndarray
    expert_nrep: np.ndarray
    expert_rep_weight: Optional[np.ndarray]
    slot_widx: np.ndarray
    slot_gidx: np.ndarray
    local_experts: np.ndarray
    # per-source split (Sec. 7.2 r_{s,e,j} per source rank): source s owns
    # tokens [src_token_begin[s], src_token_begin[s+1]); src_rep_weight
    # [n_src, E, R_max] integer weights (None = the per-expert ones)
    src_token_begin: Optional[np.ndarray] = None
    src_rep_weight: Optional[np.ndarray] = None

    @property
    def n_src(self) -> int:
        return 1 if self.src_token_begin is None else int(len(self.src_token_begin) - 1)

    @property
    def S(self) -> int:
        return int(self.slot_expert.shape[0])

    @property
    def W(self) -> int:
        return int(self.local_experts.shape[0])

    @property
    def G(self) -> int:
        return int(self.local_experts.shape[0])


def plan_from_slots(E: int, slots: Sequence[Tuple[int, int]],
                    nrep: Optional[Dict[int, int]] = None,
                    rep_weights: Optional[Dict[int, Sequence[int]]] = None,
                    R_max: Optional[int] = None) -> Plan:
    """Build a Plan from a list of (expert, replica) slots.

    ``nrep[e]`` defaults to 1 + the largest local replica index of e (1 for
    experts with no local slot). ``rep_weights[e]`` gives integer split
    weights for the replicas of e (others split equally).
    """
    slots = [(int(e), int(r)) for e, r in slots]
    nr = np.ones(E, dtype=np.int32)
    for e, r in slots:
        nr[e] = max(nr[e], r + 1)
    if nrep:
        for e, R in nrep.items():
            nr[e] = int(R)
    rmax = int(R_max) if R_max is not None else int(nr.max())
    if rmax < int(nr.max()):
        raise ValueError("R_max below a replica count")
    weights = None
    if rep_weights:
        weights = np.zeros((E, rmax), dtype=np.int32)
        for e in range(E):
            weights[e, :nr[e]] = 1
        for e, w in rep_weights.items():
            if len(w) != nr[e]:
                raise ValueError("one weight per replica expected")
            weights[e, :nr[e]] = np.asarray(w, dtype=np.int32)
    local: List[int] = []
    for e, _ in slots:
        if e not in local:
            local.append(e)
    widx = np.array([local.index(e) for e, _ in slots], dtype=np.int32)
    return Plan(E=E, R_max=rmax,
                slot_expert=np.array([e for e, _ in slots], dtype=np.int32),
                slot_replica=np.array([r for _, r in slots], dtype=np.int32),
                expert_nrep=nr, expert_rep_weight=weights,
                slot_widx=widx, slot_gidx=widx.copy(),
                local_experts=np.array(local, dtype=np.int32))


@dataclass
class MicroStep:
    index: int
    ids: np.ndarray       # int32 [T, K]
    gates: np.ndarray     # float32 [T, K]
    plan: Plan
    expert_load: np.ndarray  # int64 [E] foreseen load (planner input)


@dataclass
class Workload:
    spec: ConfigSpec
    micro: List[MicroStep]
    measured: int
    rank: int
    base_rank_of_expert: np.ndarray
    stats: Dict[str, float] = field(default_factory=dict)
    _cache: Dict[str, np.ndarray] = field(default_factory=dict, repr=False)

    def _seq(self, *key: int) -> np.random.Generator:
        return np.random.default_rng(np.random.SeedSequence(self.spec.seed, spawn_key=key))

    def _round(self, a: np.ndarray) -> np.ndarray:
        return bf16_round(a) if self.spec.dtype == "bf16" else a.astype(np.float32)

    def x(self, i: int) -> np.ndarray:
        """Token activations [T, d], N(0,1)."""
        key = f"x{i}"
        if key not in self._cache:
            rng = self._seq(1 + i, 1)
            self._cache[key] = self._round(rng.standard_normal((self.spec.T, self.spec.d), dtype=np.float32))
        return self._cache[key]

    def dy(self, i: int) -> np.ndarray:
        """Upstream gradient of the layer output [T, d], N(0,1)."""
        key = f"dy{i}"
        if key not in self._cache:
            rng = self._seq(1 + i, 2)
            self._cache[key] = self._round(rng.standard_normal((self.spec.T, self.spec.d), dtype=np.float32))
        return self._cache[key]

    def expert_weights(self, e: int) -> Tuple[np.ndarray, np.ndarray]:
        """Weights of global expert e: gate/up stacked [2F, d] and down [d, F].

        Gate and up ~ N(0, 1/d) (variance 1/fan-in); down ~ N(0, 1/F).
        """
        key = f"w{e}"
        if key not in self._cache:
            s = self.spec
            rng = self._seq(0, 1 + e)
            gu = rng.standard_normal((2 * s.F, s.d), dtype=np.float32) * np.float32(1.0 / np.sqrt(s.d))
            dn = rng.standard_normal((s.d, s.F), dtype=np.float32) * np.float32(1.0 / np.sqrt(s.F))
            self._cache[key] = (self._round(gu), self._round(dn))
        return self._cache[key]

    def weights(self, plan: Plan) -> Tuple[np.ndarray, np.ndarray]:
        """Stacked weights of the plan's local experts: [W, 2F, d] and [W, d, F]."""
        gu = np.stack([self.expert_weights(int(e))[0] for e in plan.local_experts])
        dn = np.stack([self.expert_weights(int(e))[1] for e in plan.local_experts])
        return gu, dn


def _popularity(spec: ConfigSpec) -> np.ndarray:
    rank = np.arange(spec.E)
    if spec.permute_popularity:
        rng = np.random.default_rng(np.random.SeedSequence(spec.seed, spawn_key=(0, 0)))
        rank = rng.permutation(spec.E)
    return (rank.astype(np.float64) + 1.0) ** (-spec.zipf_s)


def _routing(spec: ConfigSpec, z: np.ndarray, i: int) -> Tuple[np.ndarray, np.ndarray]:
    rng = np.random.default_rng(np.random.SeedSequence(spec.seed, spawn_key=(1 + i, 0)))
    bias = np.log(z)
    if spec.alpha is not None:
        g = rng.dirichlet(np.full(spec.E, spec.alpha))
        bias = bias + np.log(np.maximum(spec.E * g, 1e-30))
    logits = rng.standard_normal((spec.T, spec.E)) + bias[None, :]
    order = np.argsort(-logits, axis=1, kind="stable")
    ids = order[:, :spec.K].astype(np.int32)
    m = logits.max(axis=1, keepdims=True)
    p = np.exp(logits - m)
    p /= p.sum(axis=1, keepdims=True)
    sel = np.take_along_axis(p, ids.astype(np.int64), axis=1)
    gates = (sel / sel.sum(axis=1, keepdims=True)).astype(np.float32)
    return ids, gates


def _load(ids: np.ndarray, E: int) -> np.ndarray:
    """Foreseen per-expert load of a micro-step (the planner's input)."""
    return np.bincount(ids.reshape(-1), minlength=E).astype(np.int64)


def _lpt_base_placement(load: np.ndarray, P: int) -> np.ndarray:
    """Rank-level LPT of Alg. 1 (one machine) with E/P base slots per rank."""
    E = load.shape[0]
    cap = E // P
    order = np.argsort(-load, kind="stable")
    rl = np.zeros(P, dtype=np.int64)
    used = np.zeros(P, dtype=np.int64)
    place = np.full(E, -1, dtype=np.int64)
    for e in order:
        best = -1
        for r in range(P):
            if used[r] < cap and (best < 0 or rl[r] < rl[best]):
                best = r
        place[e] = best
        rl[best] += load[e]
        used[best] += 1
    return place


def _share_plan(spec: ConfigSpec, hosted: np.ndarray, load: np.ndarray) -> Plan:
    hosted = np.sort(hosted)
    hl = load[hosted]
    order = np.argsort(-hl, kind="stable")[: spec.n_rep]
    reps = hosted[order]
    slots = [(int(e), 0) for e in hosted] + [(int(e), 1) for e in reps]
    return plan_from_slots(spec.E, slots, R_max=2)


def make_workload(spec_or_id, micro_steps: Optional[int] = None) -> Workload:
    """Generate the routing, plans and lazily-drawn values of a workload, given
    by its spec, its name or its id in the table."""
    if isinstance(spec_or_id, str):
        spec_or_id = CONFIG_IDS[spec_or_id]
    spec = CONFIGS[spec_or_id] if isinstance(spec_or_id, int) else spec_or_id
    n_micro = spec.micro_steps if micro_steps is None else micro_steps
    z = _popularity(spec)
    routing = [_routing(spec, z, i) for i in range(n_micro)]
    loads = [_load(ids, spec.E) for ids, _ in routing]
    stats: Dict[str, float] = {}

    if spec.cid == 1 and spec.P == 1 and spec.E == 8:
        # Four local slots: experts 0, 1, 2 and a second replica of expert 0.
        plan = plan_from_slots(spec.E, [(0, 0), (1, 0), (2, 0), (0, 1)], R_max=2)
        micro = [MicroStep(i, ids, g, plan, loads[i]) for i, (ids, g) in enumerate(routing)]
        return Workload(spec, micro, 0, 0, np.zeros(spec.E, dtype=np.int64), stats)

    if spec.P == 1:
        base = np.zeros(spec.E, dtype=np.int64)
        rank = 0
    else:
        agg = np.sum(loads, axis=0)
        base = _lpt_base_placement(agg, spec.P)
        rank_load = np.bincount(base, weights=agg, minlength=spec.P)
        mean = rank_load.mean()
        rank = int(np.argmin(np.abs(rank_load - mean)))
        seq_load = np.bincount(np.arange(spec.E) // (spec.E // spec.P), weights=agg, minlength=spec.P)
        stats["imbalance_sequential"] = float(seq_load.max() / seq_load.mean())
        stats["imbalance_lpt"] = float(rank_load.max() / rank_load.mean())
    hosted = np.nonzero(base == rank)[0]
    micro = []
    for i, (ids, g) in enumerate(routing):
        micro.append(MicroStep(i, ids, g, _share_plan(spec, hosted, loads[i]), loads[i]))
    local_pairs = np.array([int(loads[i][hosted].sum()) for i in range(n_micro)])
    target = spec.T * spec.K / spec.P
    measured = int(np.argmin(np.abs(local_pairs - target)))
    stats["local_pairs_measured"] = float(local_pairs[measured])
    stats["local_pairs_median"] = float(np.median(local_pairs))
    stats["local_pairs_min"] = float(local_pairs.min())
    stats["local_pairs_max"] = float(local_pairs.max())
    return Workload(spec, micro, measured, rank, base, stats)


def make_custom(T: int, d: int, F: int, E: int, K: int, dtype: str = "bf16", *,
                zipf_s: float = 1.1, alpha: Optional[float] = 0.3, P: int = 1,
                n_rep: int = 1, micro_steps: int = 1, seed: int = 7,
                permute_popularity: bool = True) -> Workload:
    """A workload of arbitrary shape drawn with the same recipe (for tests)."""
    spec = ConfigSpec(0, f"custom-T{T}-d{d}-F{F}-E{E}-K{K}", T=T, d=d, F=F, E=E, K=K,
                      dtype=dtype, zipf_s=zipf_s, alpha=alpha,
                      permute_popularity=permute_popularity, P=P, n_rep=n_rep,
                      micro_steps=micro_steps, backward=True, seed=seed)
    return make_workload(spec)
