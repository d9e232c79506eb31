"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI
(via the thin binding) and the fp64 oracle on the same seeded inputs."""
from __future__ import annotations

import functools

import numpy as np
import torch

import oracle.foremoe_oracle as O
from workload import bf16_round, make_custom, make_workload

TOL_REL = 1e-2
TOL_ABS = 1e-3


def check_close(name: str, got, ref) -> None:
    """max|err| <= 1e-2 * max|ref| + 1e-3 over the whole tensor."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, f"{name}: shape {got.shape} vs {ref.shape}"
    assert np.all(np.isfinite(got)), f"{name}: non-finite values"
    err = float(np.max(np.abs(got - ref))) if got.size else 0.0
    bound = TOL_REL * (float(np.max(np.abs(ref))) if ref.size else 0.0) + TOL_ABS
    assert err <= bound, f"{name}: max|err| {err:.4g} > {bound:.4g}"


def tdtype(w) -> torch.dtype:
    return torch.bfloat16 if w.spec.dtype == "bf16" else torch.float32


def to_dev(a, dtype, dev) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev).to(dtype)


def to_np(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def rnd(w, a):
    """Round an oracle value to the storage precision of the workload."""
    return bf16_round(np.asarray(a, dtype=np.float32)) if w.spec.dtype == "bf16" else np.asarray(a, np.float32)


@functools.lru_cache(maxsize=None)
def config_workload(name: str):
    return make_workload(name)


@functools.lru_cache(maxsize=None)
def custom_workload(name: str):
    shapes = {
        # several 256-row tiles, ragged tails, 256-wide output tiles
        "small": dict(T=1024, d=256, F=256, E=8, K=2, P=1, n_rep=2, seed=31),
        # d and F not multiples of 256: 128-wide output tiles
        "odd128": dict(T=768, d=384, F=384, E=6, K=2, P=1, n_rep=2, seed=32),
        # EP share with empty slots and skew, as the RL configs
        "share": dict(T=2048, d=256, F=128, E=32, K=4, P=4, n_rep=2, seed=33, micro_steps=4),
        "tinyf32": dict(T=96, d=24, F=40, E=5, K=2, P=1, n_rep=1, seed=34, dtype="f32"),
    }
    return make_custom(**shapes[name])


def gpu_dispatch(w, m, dev, n_cap=None, x=None, fused=True):
    """Steps 1-3 on the GPU; returns device tensors and the workspace.
    fused: steps 1-2 through foremoe_histogram_assign (as the benchmark runs
    them), else through foremoe_histogram and foremoe_assign_replicas."""
    from paper_2606_11867_amd import api
    T, K = m.ids.shape
    if n_cap is None:
        n_cap = T * K
    if x is None:
        x = w.x(m.index)
    ids = torch.from_numpy(m.ids).to(dev)
    plan = api.DevicePlan.from_host(m.plan, dev)
    ws = api.workspace(T, K, m.plan.E, dev)
    if fused:
        counts, rep_begin, slot_count, slot_offset = api.histogram_assign(ids, plan, ws)
    else:
        counts = api.histogram(ids, m.plan.E, ws)
        rep_begin, slot_count, slot_offset = api.assign_replicas(counts, plan, ws)
    xd = to_dev(x, tdtype(w), dev)
    x_perm, r2p, p2r = api.permute(xd, ids, plan, rep_begin, slot_offset, n_cap, ws)
    return dict(ids=ids, plan=plan, ws=ws, counts=counts, rep_begin=rep_begin, slot_count=slot_count,
                slot_offset=slot_offset, x=xd, x_perm=x_perm, row_to_pair=r2p, pair_to_row=p2r, n_cap=n_cap)


def oracle_dispatch(w, m, n_cap=None, x=None):
    T, K = m.ids.shape
    if n_cap is None:
        n_cap = T * K
    if x is None:
        x = w.x(m.index)
    counts, invalid = O.histogram(m.ids, m.plan.E)
    rep_begin, slot_count, slot_offset = O.assign_replicas(counts, m.plan)
    x_perm, r2p, p2r, dropped = O.permute(x, m.ids, m.plan, rep_begin, slot_offset, n_cap)
    return dict(counts=counts, invalid=invalid, rep_begin=rep_begin, slot_count=slot_count,
                slot_offset=slot_offset, x_perm=x_perm, row_to_pair=r2p, pair_to_row=p2r, dropped=dropped)
