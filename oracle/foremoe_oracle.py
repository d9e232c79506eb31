"""Plain fp64 CPU oracle of the per-micro-step MoE expert layer.

TEST INFRASTRUCTURE. Only tests/, the smoke check and the benchmark's CPU
baseline may import or run this module; the product path never does.

What it computes is the plain MoE layer of the paper (Sec. 2.1): every token
is sent to its top-K experts and the layer output is the router-probability
weighted sum of those experts' outputs. ForeMoE's placement (Sec. 7) only
changes *where* a (token, k) pair is computed: expert replicas hold the same
weights, and the token-conservation and feasibility constraints of the MILP
(Sec. 7.2, App. C) say that every pair of an expert is processed by exactly
one slot that holds that expert. So the oracle is that definition written out
step by step for one GPU's slots, in float64, with no blocking or fusion:

1. histogram  - tokens per expert from the recorded top-K ids (Sec. 5,
                Routing Collector; load w_{s,e} of Table 1);
2. assign     - contiguous split of each expert's token list over its
                replicas in the proportions of the token-assignment fractions
                r_{s,e,j} (Sec. 7.2; Sec. 8 Stage 4; App. D Stage 4);
3. permute    - gather tokens into slot-contiguous order;
4. grouped FFN- SwiGLU expert with gate, up and down matrices (App. A,
                Eq. flops_moe) per slot; backward by the chain rule, with the
                weight gradients of all replicas of an expert summed into one
                main-expert gradient (Sec. 6.2, Copy-in);
5. combine    - gate-weighted sum back to token order (Sec. 2.1).

Readings where the paper is silent (stated once here, used throughout):
* the token list of expert e is the pairs p = t*K + k with ids[p] == e in
  ascending p; replica r of e takes the contiguous block
  [floor(n_e*W_r/W), floor(n_e*W_{r+1}/W)) where W_r is the prefix sum of the
  integer split weights (equal weights give floor(r*n_e/R_e));
* id -1 is padding (skipped, not an error); other ids outside [0, E) are
  invalid (skipped and counted);
* SwiGLU is down(silu(gate x) * up x), silu(a) = a / (1 + exp(-a)), no bias;
* replica 0 of an expert is its main expert (``slot_gidx`` of every replica
  slot points at it);
* a token with no local pair gets an all-zero output row.

Floating-point inputs are taken as given (already rounded to bf16 or fp32 by
the generator) and everything is computed in float64.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Tuple

import numpy as np


# ----------------------------------------------------------------------------
# Step 1: histogram (recorded routing -> per-expert load)
# ----------------------------------------------------------------------------
def histogram(ids: np.ndarray, E: int) -> Tuple[np.ndarray, int]:
    """counts[e] = number of (token, k) pairs whose recorded expert is e.

    Routing record of Sec. 5 (top-K ids per token); the per-expert token
    volume is the load w_e of Table 1. Returns (counts int32 [E], invalid),
    where ``invalid`` is the number of ids outside [-1, E).
    """
    flat = np.asarray(ids).reshape(-1).astype(np.int64)
    valid = (flat >= 0) & (flat < E)
    counts = np.bincount(flat[valid], minlength=E)
    invalid = int(np.count_nonzero((flat != -1) & ~valid))
    return counts.astype(np.int32), invalid


# ----------------------------------------------------------------------------
# Step 2: replica split (token conservation, Sec. 7.2 / App. C)
# ----------------------------------------------------------------------------
def replica_bounds(n: int, weights: List[int]) -> List[int]:
    """Boundaries B[0..R] of the contiguous split of n tokens over R replicas.

    B[r] = floor(n * (w_0 + ... + w_{r-1}) / (w_0 + ... + w_{R-1})), exact
    integer arithmetic; B[0] = 0 and B[R] = n, so the blocks cover the list
    exactly once (sum_j r_{s,e,j} = 1).
    """
    total = int(sum(int(w) for w in weights))
    if total <= 0 or any(int(w) < 0 for w in weights):
        raise ValueError("replica weights must be >= 0 with a positive sum")
    out = [0]
    pref = 0
    for w in weights:
        pref += int(w)
        out.append((int(n) * pref) // total)
    return out


def assign_replicas(counts: np.ndarray, plan) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Per-replica token ranges and the local slots' counts and offsets.

    Returns rep_begin int32 [E, R_max+1] (entries past R_e hold n_e),
    slot_count int32 [S] and slot_offset int32 [S+1] (exclusive prefix sum of
    slot_count in slot-table order; slot_offset[S] = N local pairs).
    """
    E, R_max = plan.E, plan.R_max
    rep_begin = np.zeros((E, R_max + 1), dtype=np.int64)
    for e in range(E):
        R = int(plan.expert_nrep[e])
        if plan.expert_rep_weight is None:
            w = [1] * R
        else:
            w = [int(v) for v in np.asarray(plan.expert_rep_weight).reshape(E, R_max)[e, :R]]
        b = replica_bounds(int(counts[e]), w)
        rep_begin[e, : R + 1] = b
        rep_begin[e, R + 1:] = int(counts[e])
    S = plan.S
    slot_count = np.zeros(S, dtype=np.int64)
    for j in range(S):
        e, r = int(plan.slot_expert[j]), int(plan.slot_replica[j])
        slot_count[j] = rep_begin[e, r + 1] - rep_begin[e, r]
    slot_offset = np.zeros(S + 1, dtype=np.int64)
    for j in range(S):
        slot_offset[j + 1] = slot_offset[j] + slot_count[j]
    return rep_begin.astype(np.int32), slot_count.astype(np.int32), slot_offset.astype(np.int32)


# ----------------------------------------------------------------------------
# Steps 1-2 per source rank (Sec. 7.2: r_{s,e,j} is a fraction per source
# rank s; App. D Stage 4 water-fills source by source)
# ----------------------------------------------------------------------------
# Reading: source rank s owns the contiguous tokens [tb[s], tb[s+1]) of the
# micro-step; for each (s, e) the pairs of s routed to e, in ascending p,
# are split over e's replicas by the weights of (s, e) with the same floor
# rule as above; a replica's slot takes its blocks source by source, so the
# rows of a slot stay in ascending p. All-zero weights are an error only
# when (s, e) has pairs (a planner gives zero weights to empty pairs).
def histogram_src(ids: np.ndarray, E: int, src_token_begin) -> np.ndarray:
    """counts[s, e] = #pairs of tokens of source s with ids == e."""
    ids = np.asarray(ids)
    tb = [int(v) for v in src_token_begin]
    out = np.zeros((len(tb) - 1, E), dtype=np.int32)
    for s in range(len(tb) - 1):
        out[s], _ = histogram(ids[tb[s]:tb[s + 1]], E)
    return out


def _src_weights(plan, s: int, e: int, R: int) -> List[int]:
    if getattr(plan, "src_rep_weight", None) is not None:
        return [int(v) for v in np.asarray(plan.src_rep_weight)[s, e, :R]]
    if plan.expert_rep_weight is not None:
        return [int(v) for v in np.asarray(plan.expert_rep_weight).reshape(plan.E, plan.R_max)[e, :R]]
    return [1] * R


def assign_replicas_src(counts_src: np.ndarray, plan) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Per-(source, expert) replica ranges and the local slots' counts/offsets.

    Returns rep_begin int32 [n_src, E, R_max+1] (entries past R_e hold n_{s,e}),
    slot_count int32 [S] (summed over sources) and slot_offset int32 [S+1].
    """
    counts_src = np.asarray(counts_src)
    n_src, E = counts_src.shape
    R_max = plan.R_max
    rep_begin = np.zeros((n_src, E, R_max + 1), dtype=np.int64)
    for s in range(n_src):
        for e in range(E):
            R = int(plan.expert_nrep[e])
            n = int(counts_src[s, e])
            w = _src_weights(plan, s, e, R)
            b = replica_bounds(n, w) if sum(w) > 0 else replica_bounds(n, [1] * R)
            rep_begin[s, e, : R + 1] = b
            rep_begin[s, e, R + 1:] = n
    slot_count = np.zeros(plan.S, dtype=np.int64)
    for j in range(plan.S):
        e, r = int(plan.slot_expert[j]), int(plan.slot_replica[j])
        slot_count[j] = int(np.sum(rep_begin[:, e, r + 1] - rep_begin[:, e, r]))
    slot_offset = np.zeros(plan.S + 1, dtype=np.int64)
    for j in range(plan.S):
        slot_offset[j + 1] = slot_offset[j] + slot_count[j]
    return rep_begin.astype(np.int32), slot_count.astype(np.int32), slot_offset.astype(np.int32)


def permute_src(x: np.ndarray, ids: np.ndarray, plan, rep_begin_src: np.ndarray, slot_offset: np.ndarray,
                n_cap: int, src_token_begin):
    """permute() with per-source replica ranges: slot j holds, source by
    source, the pairs of its replica's block in each source's list."""
    ids = np.asarray(ids)
    T, K = ids.shape
    tb = [int(v) for v in src_token_begin]
    d = x.shape[1]
    x_perm = np.zeros((n_cap, d), dtype=np.float64)
    row_to_pair = np.full(n_cap, -1, dtype=np.int32)
    pair_to_row = np.full(T * K, -1, dtype=np.int32)
    dropped = 0
    for j in range(plan.S):
        e, r = int(plan.slot_expert[j]), int(plan.slot_replica[j])
        row = int(slot_offset[j])
        for s in range(len(tb) - 1):
            flat = ids[tb[s]:tb[s + 1]].reshape(-1)
            plist = tb[s] * K + np.nonzero(flat == e)[0]   # source s's list of e, ascending p
            for p in plist[int(rep_begin_src[s, e, r]):int(rep_begin_src[s, e, r + 1])]:
                if row >= n_cap:
                    dropped += 1
                else:
                    pair_to_row[p] = row
                    row_to_pair[row] = p
                    x_perm[row] = x[p // K]
                row += 1
    return x_perm, row_to_pair, pair_to_row, dropped


# ----------------------------------------------------------------------------
# Step 3: permute (dispatch of each pair to exactly one local slot)
# ----------------------------------------------------------------------------
def permute(x: np.ndarray, ids: np.ndarray, plan, rep_begin: np.ndarray,
            slot_offset: np.ndarray, n_cap: int):
    """Gather token rows into slot-contiguous order.

    Pair p of expert e is the q-th entry of e's token list; it belongs to the
    replica r with B[r] <= q < B[r+1]. If that replica is local in slot j its
    row is slot_offset[j] + q - B[r]. Returns (x_perm [n_cap, d] float64 with
    rows >= N zero, row_to_pair int32 [n_cap] with -1 past N, pair_to_row
    int32 [T*K] with -1 for pairs not computed here, dropped) where
    ``dropped`` counts local pairs whose row would reach n_cap (those keep
    pair_to_row -1).
    """
    ids = np.asarray(ids)
    T, K = ids.shape
    flat = ids.reshape(-1)
    d = x.shape[1]
    local: Dict[Tuple[int, int], int] = {}
    for j in range(plan.S):
        local[(int(plan.slot_expert[j]), int(plan.slot_replica[j]))] = j
    x_perm = np.zeros((n_cap, d), dtype=np.float64)
    row_to_pair = np.full(n_cap, -1, dtype=np.int32)
    pair_to_row = np.full(T * K, -1, dtype=np.int32)
    dropped = 0
    for e in range(plan.E):
        plist = np.nonzero(flat == e)[0]          # ascending p: the canonical list
        R = int(plan.expert_nrep[e])
        for r in range(R):
            j = local.get((e, r))
            if j is None:
                continue
            lo, hi = int(rep_begin[e, r]), int(rep_begin[e, r + 1])
            for i in range(hi - lo):
                p = int(plist[lo + i])
                row = int(slot_offset[j]) + i
                if row >= n_cap:
                    dropped += 1
                    continue
                pair_to_row[p] = row
                row_to_pair[row] = p
                x_perm[row] = x[p // K]
    return x_perm, row_to_pair, pair_to_row, dropped


# ----------------------------------------------------------------------------
# Step 4: grouped SwiGLU FFN over local slots (App. A)
# ----------------------------------------------------------------------------
def silu(a: np.ndarray) -> np.ndarray:
    return a / (1.0 + np.exp(-a))


def _split(w_gate_up: np.ndarray, widx: int):
    F = w_gate_up.shape[1] // 2
    wg = np.asarray(w_gate_up[widx, :F], dtype=np.float64)
    wu = np.asarray(w_gate_up[widx, F:], dtype=np.float64)
    return wg, wu


def ffn_forward(x_perm: np.ndarray, slot_offset: np.ndarray, slot_widx: np.ndarray,
                w_gate_up: np.ndarray, w_down: np.ndarray) -> Dict[str, np.ndarray]:
    """Per slot j over rows [o_j, o_{j+1}): A = X Wg^T, U = X Wu^T,
    H = silu(A) * U, Y = H Wd^T. w_gate_up [W, 2F, d] holds gate rows [0, F)
    and up rows [F, 2F); w_down is [W, d, F]. Returns A, U, H, Y (float64,
    rows past N zero)."""
    n_rows, d = x_perm.shape
    F = w_gate_up.shape[1] // 2
    A = np.zeros((n_rows, F))
    U = np.zeros((n_rows, F))
    H = np.zeros((n_rows, F))
    Y = np.zeros((n_rows, d))
    for j in range(len(slot_widx)):
        lo, hi = int(slot_offset[j]), int(slot_offset[j + 1])
        if hi <= lo:
            continue
        w = int(slot_widx[j])
        wg, wu = _split(w_gate_up, w)
        wd = np.asarray(w_down[w], dtype=np.float64)
        X = np.asarray(x_perm[lo:hi], dtype=np.float64)
        A[lo:hi] = X @ wg.T
        U[lo:hi] = X @ wu.T
        H[lo:hi] = silu(A[lo:hi]) * U[lo:hi]
        Y[lo:hi] = H[lo:hi] @ wd.T
    return {"A": A, "U": U, "H": H, "Y": Y}


def ffn_dgrad(dy_perm: np.ndarray, A: np.ndarray, U: np.ndarray, slot_offset: np.ndarray,
              slot_widx: np.ndarray, w_gate_up: np.ndarray, w_down: np.ndarray) -> Dict[str, np.ndarray]:
    """Input gradients of the SwiGLU expert by the chain rule:
    dH = dY Wd, dA = dH * U * silu'(A), dU = dH * silu(A),
    dX = dA Wg + dU Wu, with silu'(a) = s + a s (1 - s), s = 1/(1+exp(-a))."""
    n_rows, d = dy_perm.shape
    F = w_gate_up.shape[1] // 2
    dA = np.zeros((n_rows, F))
    dU = np.zeros((n_rows, F))
    dX = np.zeros((n_rows, d))
    for j in range(len(slot_widx)):
        lo, hi = int(slot_offset[j]), int(slot_offset[j + 1])
        if hi <= lo:
            continue
        w = int(slot_widx[j])
        wg, wu = _split(w_gate_up, w)
        wd = np.asarray(w_down[w], dtype=np.float64)
        dY = np.asarray(dy_perm[lo:hi], dtype=np.float64)
        a = np.asarray(A[lo:hi], dtype=np.float64)
        u = np.asarray(U[lo:hi], dtype=np.float64)
        dH = dY @ wd
        s = 1.0 / (1.0 + np.exp(-a))
        dA[lo:hi] = dH * u * (s + a * s * (1.0 - s))
        dU[lo:hi] = dH * (a * s)
        dX[lo:hi] = dA[lo:hi] @ wg + dU[lo:hi] @ wu
    return {"dA": dA, "dU": dU, "dX": dX}


def ffn_wgrad(x_perm: np.ndarray, H: np.ndarray, dy_perm: np.ndarray, dA: np.ndarray,
              dU: np.ndarray, slot_offset: np.ndarray, slot_gidx: np.ndarray, G: int,
              dw_gate_up: Optional[np.ndarray] = None,
              dw_down: Optional[np.ndarray] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Weight gradients, accumulated (+=) into the main expert of each slot:
    dWg[g] += dA^T X, dWu[g] += dU^T X, dWd[g] += dY^T H over the rows of
    every slot whose gradient index is g (Sec. 6.2: replica gradients are
    summed into the main expert). Returns (dW_gate_up [G, 2F, d],
    dW_down [G, d, F]) in float64."""
    d = x_perm.shape[1]
    F = H.shape[1]
    if dw_gate_up is None:
        dw_gate_up = np.zeros((G, 2 * F, d))
    if dw_down is None:
        dw_down = np.zeros((G, d, F))
    for j in range(len(slot_gidx)):
        lo, hi = int(slot_offset[j]), int(slot_offset[j + 1])
        if hi <= lo:
            continue
        g = int(slot_gidx[j])
        X = np.asarray(x_perm[lo:hi], dtype=np.float64)
        dw_gate_up[g, :F] += np.asarray(dA[lo:hi], dtype=np.float64).T @ X
        dw_gate_up[g, F:] += np.asarray(dU[lo:hi], dtype=np.float64).T @ X
        dw_down[g] += np.asarray(dy_perm[lo:hi], dtype=np.float64).T @ np.asarray(H[lo:hi], dtype=np.float64)
    return dw_gate_up, dw_down


# ----------------------------------------------------------------------------
# Step 5: combine, and the backward gathers
# ----------------------------------------------------------------------------
def combine(y_perm: np.ndarray, pair_to_row: np.ndarray, gates: np.ndarray, T: int, K: int) -> np.ndarray:
    """y[t] = sum over k (ascending) of gates[t, k] * Y[row(t, k)] for the
    pairs computed here (Sec. 2.1); tokens with none get a zero row."""
    d = y_perm.shape[1]
    y = np.zeros((T, d))
    g = np.asarray(gates, dtype=np.float64).reshape(T, K)
    for t in range(T):
        for k in range(K):
            row = int(pair_to_row[t * K + k])
            if row >= 0:
                y[t] += g[t, k] * np.asarray(y_perm[row], dtype=np.float64)
    return y


def combine_bwd(dy: np.ndarray, y_perm: np.ndarray, row_to_pair: np.ndarray, gates: np.ndarray,
                n_rows: int, T: int, K: int) -> Tuple[np.ndarray, np.ndarray]:
    """Gradients of the combine: dY[row] = gates[p] * dy[t(p)] and
    dgates[p] = <dy[t(p)], Y[row]> for the n_rows local rows; dgates of pairs
    not computed here are 0."""
    d = dy.shape[1]
    dY = np.zeros((len(row_to_pair), d))
    dgates = np.zeros(T * K)
    g = np.asarray(gates, dtype=np.float64).reshape(-1)
    for row in range(n_rows):
        p = int(row_to_pair[row])
        t = p // K
        dyt = np.asarray(dy[t], dtype=np.float64)
        dY[row] = g[p] * dyt
        dgates[p] = float(np.dot(dyt, np.asarray(y_perm[row], dtype=np.float64)))
    return dY, dgates.reshape(T, K)


def permute_bwd(dx_perm: np.ndarray, pair_to_row: np.ndarray, T: int, K: int) -> np.ndarray:
    """dx[t] = sum over k (ascending) of dX[row(t, k)] for pairs computed here."""
    d = dx_perm.shape[1]
    dx = np.zeros((T, d))
    for t in range(T):
        for k in range(K):
            row = int(pair_to_row[t * K + k])
            if row >= 0:
                dx[t] += np.asarray(dx_perm[row], dtype=np.float64)
    return dx


# ----------------------------------------------------------------------------
# The whole layer, step after step
# ----------------------------------------------------------------------------
def layer_forward(x, ids, gates, plan, w_gate_up, w_down, n_cap: Optional[int] = None) -> Dict:
    """Steps 1-5 in order for one micro-step; returns every intermediate."""
    ids = np.asarray(ids)
    T, K = ids.shape
    if n_cap is None:
        n_cap = T * K
    counts, invalid = histogram(ids, plan.E)
    rep_begin, slot_count, slot_offset = assign_replicas(counts, plan)
    x_perm, row_to_pair, pair_to_row, dropped = permute(x, ids, plan, rep_begin, slot_offset, n_cap)
    f = ffn_forward(x_perm, slot_offset, plan.slot_widx, w_gate_up, w_down)
    y = combine(f["Y"], pair_to_row, gates, T, K)
    out = dict(counts=counts, invalid=invalid, rep_begin=rep_begin, slot_count=slot_count,
               slot_offset=slot_offset, x_perm=x_perm, row_to_pair=row_to_pair,
               pair_to_row=pair_to_row, dropped=dropped, y=y)
    out.update(f)
    return out


def layer_backward(fwd: Dict, dy, gates, plan, w_gate_up, w_down, T: int, K: int,
                   dw_gate_up: Optional[np.ndarray] = None,
                   dw_down: Optional[np.ndarray] = None) -> Dict:
    """Backward of one micro-step with the forward's plan (Sec. 6.2: the plan
    is retained for the backward). Weight gradients accumulate (+=)."""
    n_rows = int(fwd["slot_offset"][-1])
    dY, dgates = combine_bwd(dy, fwd["Y"], fwd["row_to_pair"], gates, n_rows, T, K)
    g = ffn_dgrad(dY, fwd["A"], fwd["U"], fwd["slot_offset"], plan.slot_widx, w_gate_up, w_down)
    dwgu, dwd = ffn_wgrad(fwd["x_perm"], fwd["H"], dY, g["dA"], g["dU"], fwd["slot_offset"],
                          plan.slot_gidx, plan.G, dw_gate_up, dw_down)
    dx = permute_bwd(g["dX"], fwd["pair_to_row"], T, K)
    return dict(dy_perm=dY, dgates=dgates, dA=g["dA"], dU=g["dU"], dx_perm=g["dX"], dx=dx,
                dw_gate_up=dwgu, dw_down=dwd)
