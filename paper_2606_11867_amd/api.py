"""Tensor-level binding of the C ABI: argument marshalling only.

Every function allocates its outputs with torch (device memory), passes raw
device pointers and the current HIP stream to libforemoe.so and raises if the
library reports an error. No arithmetic of the expert layer happens here.
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass
from typing import Optional, Tuple

import numpy as np
import torch

from . import _lib
from ._lib import check

_DT = {torch.float32: _lib.F32, torch.bfloat16: _lib.BF16}


def _dt(t: torch.Tensor) -> int:
    if t.dtype not in _DT:
        raise TypeError(f"unsupported dtype {t.dtype}")
    return _DT[t.dtype]


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return t.data_ptr()


def _stream(device: torch.device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _i32(t: torch.Tensor, name: str) -> torch.Tensor:
    if t.dtype != torch.int32:
        raise TypeError(f"{name} must be int32")
    return t


@dataclass
class DevicePlan:
    """A slot table (see include/foremoe.h, foremoe_plan) resident on the device."""
    E: int
    S: int
    R_max: int
    W: int
    G: int
    slot_expert: torch.Tensor
    slot_replica: torch.Tensor
    expert_nrep: torch.Tensor
    expert_rep_weight: Optional[torch.Tensor]
    slot_widx: torch.Tensor
    slot_gidx: torch.Tensor
    n_src: int = 1
    src_token_begin: Optional[torch.Tensor] = None
    src_rep_weight: Optional[torch.Tensor] = None

    @classmethod
    def from_host(cls, plan, device) -> "DevicePlan":
        dev = torch.device(device)

        def t(a):
            return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)

        def opt(a):
            return None if a is None else t(np.asarray(a).reshape(-1))

        tb = getattr(plan, "src_token_begin", None)
        return cls(E=plan.E, S=plan.S, R_max=plan.R_max, W=plan.W, G=plan.G,
                   slot_expert=t(plan.slot_expert), slot_replica=t(plan.slot_replica),
                   expert_nrep=t(plan.expert_nrep), expert_rep_weight=opt(plan.expert_rep_weight),
                   slot_widx=t(plan.slot_widx), slot_gidx=t(plan.slot_gidx),
                   n_src=1 if tb is None else len(tb) - 1, src_token_begin=opt(tb),
                   src_rep_weight=opt(getattr(plan, "src_rep_weight", None)))

    def c_struct(self) -> _lib.Plan:
        def p(x):
            return None if x is None else x.data_ptr()

        return _lib.Plan(self.E, self.S, self.R_max, self.n_src, self.slot_expert.data_ptr(),
                         self.slot_replica.data_ptr(), self.expert_nrep.data_ptr(), p(self.expert_rep_weight),
                         self.slot_widx.data_ptr(), self.slot_gidx.data_ptr(), p(self.src_token_begin),
                         p(self.src_rep_weight))


def workspace(T: int, K: int, E: int, device) -> torch.Tensor:
    n = _lib.load().foremoe_workspace_size(T, K, E)
    if n == 0:
        raise ValueError("invalid workspace sizes")
    # zero-filled so that the status words read 0 before the first call
    return torch.zeros(n, dtype=torch.uint8, device=device)


def ws_status(ws: torch.Tensor) -> np.ndarray:
    """The int32 status words at the head of a workspace (synchronises)."""
    return ws[:256].view(torch.int32).cpu().numpy()


def histogram(ids: torch.Tensor, E: int, ws: torch.Tensor) -> torch.Tensor:
    _i32(ids, "ids")
    T, K = ids.shape
    counts = torch.empty(E, dtype=torch.int32, device=ids.device)
    check(_lib.load().foremoe_histogram(_ptr(ids), T, K, E, _ptr(counts), _ptr(ws), ws.numel(),
                                        _stream(ids.device)), "foremoe_histogram")
    return counts


def histogram_src(ids: torch.Tensor, E: int, src_token_begin: torch.Tensor, ws: torch.Tensor) -> torch.Tensor:
    """Per-source counts [n_src, E] (src_token_begin: device int32 [n_src + 1])."""
    _i32(ids, "ids")
    _i32(src_token_begin, "src_token_begin")
    T, K = ids.shape
    n_src = src_token_begin.numel() - 1
    counts = torch.empty((n_src, E), dtype=torch.int32, device=ids.device)
    check(_lib.load().foremoe_histogram_src(_ptr(ids), T, K, E, n_src, _ptr(src_token_begin), _ptr(counts), _ptr(ws),
                                            ws.numel(), _stream(ids.device)), "foremoe_histogram_src")
    return counts


def assign_replicas(counts: torch.Tensor, plan: DevicePlan, ws: torch.Tensor):
    dev = counts.device
    shape = (plan.E, plan.R_max + 1) if plan.n_src <= 1 else (plan.n_src, plan.E, plan.R_max + 1)
    rep_begin = torch.empty(shape, dtype=torch.int32, device=dev)
    slot_count = torch.empty(max(plan.S, 1), dtype=torch.int32, device=dev)[: plan.S]
    slot_offset = torch.empty(plan.S + 1, dtype=torch.int32, device=dev)
    cp = plan.c_struct()
    check(_lib.load().foremoe_assign_replicas(_ptr(counts), ctypes.byref(cp), _ptr(rep_begin),
                                              slot_count.data_ptr(), _ptr(slot_offset), _ptr(ws), ws.numel(),
                                              _stream(dev)), "foremoe_assign_replicas")
    return rep_begin, slot_count, slot_offset


def histogram_assign(ids: torch.Tensor, plan: DevicePlan, ws: torch.Tensor):
    """Steps 1 and 2 in one call (two launches for up to 256 keys): the
    per-key counts (n_src * E keys for a per-source plan) and the replica
    split, as histogram(_src) followed by assign_replicas."""
    T, K = ids.shape
    dev = ids.device
    nkeys = plan.E * max(plan.n_src, 1)
    counts = torch.empty(nkeys, dtype=torch.int32, device=dev)
    shape = (plan.E, plan.R_max + 1) if plan.n_src <= 1 else (plan.n_src, plan.E, plan.R_max + 1)
    rep_begin = torch.empty(shape, dtype=torch.int32, device=dev)
    slot_count = torch.empty(max(plan.S, 1), dtype=torch.int32, device=dev)[: plan.S]
    slot_offset = torch.empty(plan.S + 1, dtype=torch.int32, device=dev)
    cp = plan.c_struct()
    check(_lib.load().foremoe_histogram_assign(_ptr(ids), T, K, ctypes.byref(cp), _ptr(counts), _ptr(rep_begin),
                                               slot_count.data_ptr(), _ptr(slot_offset), _ptr(ws), ws.numel(),
                                               _stream(dev)), "foremoe_histogram_assign")
    return counts, rep_begin, slot_count, slot_offset


def permute(x: torch.Tensor, ids: torch.Tensor, plan: DevicePlan, rep_begin: torch.Tensor,
            slot_offset: torch.Tensor, n_cap: int, ws: torch.Tensor):
    T, d = x.shape
    K = ids.shape[1]
    dev = x.device
    x_perm = torch.empty((n_cap, d), dtype=x.dtype, device=dev)
    row_to_pair = torch.empty(n_cap, dtype=torch.int32, device=dev)
    pair_to_row = torch.empty(T * K, dtype=torch.int32, device=dev)
    cp = plan.c_struct()
    check(_lib.load().foremoe_permute(_ptr(x), _dt(x), T, d, _ptr(ids), K, ctypes.byref(cp), _ptr(rep_begin),
                                      _ptr(slot_offset), n_cap, x_perm.data_ptr(), row_to_pair.data_ptr(),
                                      pair_to_row.data_ptr(), _ptr(ws), ws.numel(), _stream(dev)),
          "foremoe_permute")
    return x_perm, row_to_pair, pair_to_row


def dispatch_static(x: torch.Tensor, ids: torch.Tensor, plan: DevicePlan, n_cap: int):
    """Steps 1-3 (as histogram_assign + permute) with the library's static
    device scratch instead of a workspace; the C call allocates nothing.
    Returns counts, rep_begin, slot_count, slot_offset, x_perm, row_to_pair,
    pair_to_row and the three status words (device tensors)."""
    T, d = x.shape
    K = ids.shape[1]
    dev = x.device
    nkeys = plan.E * max(plan.n_src, 1)
    shape = (plan.E, plan.R_max + 1) if plan.n_src <= 1 else (plan.n_src, plan.E, plan.R_max + 1)
    counts = torch.empty(nkeys, dtype=torch.int32, device=dev)
    rep_begin = torch.empty(shape, dtype=torch.int32, device=dev)
    slot_count = torch.empty(max(plan.S, 1), dtype=torch.int32, device=dev)[: plan.S]
    slot_offset = torch.empty(plan.S + 1, dtype=torch.int32, device=dev)
    x_perm = torch.empty((n_cap, d), dtype=x.dtype, device=dev)
    row_to_pair = torch.empty(n_cap, dtype=torch.int32, device=dev)
    pair_to_row = torch.empty(T * K, dtype=torch.int32, device=dev)
    status = torch.empty(3, dtype=torch.int32, device=dev)
    cp = plan.c_struct()
    check(_lib.load().foremoe_dispatch_static(_ptr(ids), T, K, ctypes.byref(cp), _ptr(x), _dt(x), d, n_cap,
                                              _ptr(counts), _ptr(rep_begin), slot_count.data_ptr(),
                                              _ptr(slot_offset), x_perm.data_ptr(), row_to_pair.data_ptr(),
                                              pair_to_row.data_ptr(), _ptr(status), _stream(dev)),
          "foremoe_dispatch_static")
    return counts, rep_begin, slot_count, slot_offset, x_perm, row_to_pair, pair_to_row, status


def ffn_workspace(device) -> torch.Tensor:
    """Scratch that lets the row GEMMs cut a partial last round of tiles
    along K (foremoe_ffn_workspace_size() bytes for the current device).
    Zero-filled here, as its arrival counters must be before first use; each
    call leaves them zero again."""
    n = _lib.load().foremoe_ffn_workspace_size()
    return torch.zeros(n, dtype=torch.uint8, device=device)


def _ws(ws: Optional[torch.Tensor]):
    return (None, 0) if ws is None else (ws.data_ptr(), ws.numel())


def grouped_ffn_fwd(x_perm: torch.Tensor, slot_offset: torch.Tensor, slot_widx: torch.Tensor,
                    w_gate_up: torch.Tensor, w_down: torch.Tensor, save: bool = True,
                    ws: Optional[torch.Tensor] = None):
    n_cap, d = x_perm.shape
    W, F2, _ = w_gate_up.shape
    F = F2 // 2
    S = slot_widx.shape[0]
    dev = x_perm.device
    h = torch.empty((n_cap, F), dtype=x_perm.dtype, device=dev)
    y_perm = torch.empty((n_cap, d), dtype=x_perm.dtype, device=dev)
    save_au = torch.empty((n_cap, 2 * F), dtype=x_perm.dtype, device=dev) if save else None
    check(_lib.load().foremoe_grouped_ffn_fwd(_ptr(x_perm), _dt(x_perm), d, F, S, _ptr(slot_offset),
                                              _ptr(slot_widx), W, _ptr(w_gate_up), _ptr(w_down), n_cap,
                                              h.data_ptr(), y_perm.data_ptr(),
                                              None if save_au is None else save_au.data_ptr(), *_ws(ws),
                                              _stream(dev)),
          "foremoe_grouped_ffn_fwd")
    return h, y_perm, save_au


def grouped_ffn_dgrad(dy_perm: torch.Tensor, save_au: torch.Tensor, slot_offset: torch.Tensor,
                      slot_widx: torch.Tensor, w_gate_up: torch.Tensor, w_down: torch.Tensor,
                      ws: Optional[torch.Tensor] = None):
    n_cap, d = dy_perm.shape
    W, F2, _ = w_gate_up.shape
    F = F2 // 2
    S = slot_widx.shape[0]
    dev = dy_perm.device
    d_au = torch.empty((n_cap, 2 * F), dtype=dy_perm.dtype, device=dev)
    dx_perm = torch.empty((n_cap, d), dtype=dy_perm.dtype, device=dev)
    check(_lib.load().foremoe_grouped_ffn_dgrad(_ptr(dy_perm), _ptr(save_au), _dt(dy_perm), d, F, S,
                                                _ptr(slot_offset), _ptr(slot_widx), W, _ptr(w_gate_up),
                                                _ptr(w_down), n_cap, d_au.data_ptr(), dx_perm.data_ptr(),
                                                *_ws(ws), _stream(dev)), "foremoe_grouped_ffn_dgrad")
    return d_au, dx_perm


def wgrad_workspace(d: int, F: int, device) -> torch.Tensor:
    """Scratch for scheduling and splitting the weight-gradient work over many
    CUs. Zero-filled here, as its work-counter header must be before first
    use; each call leaves that header zero again."""
    n = _lib.load().foremoe_wgrad_workspace_size(d, F)
    return torch.zeros(n, dtype=torch.uint8, device=device)


def grouped_ffn_wgrad(x_perm: torch.Tensor, h: torch.Tensor, dy_perm: torch.Tensor, d_au: torch.Tensor,
                      slot_offset: torch.Tensor, slot_gidx: torch.Tensor, dw_gate_up: torch.Tensor,
                      dw_down: torch.Tensor, ws: Optional[torch.Tensor] = None) -> None:
    """Accumulates (+=) into the fp32 gradients dw_gate_up [G, 2F, d], dw_down [G, d, F].

    ``ws`` (from ``wgrad_workspace``) lets the kernels split skewed experts
    over many CUs; without it the result is the same, only slower."""
    n_cap, d = x_perm.shape
    G, F2, _ = dw_gate_up.shape
    F = F2 // 2
    S = slot_gidx.shape[0]
    if dw_gate_up.dtype != torch.float32 or dw_down.dtype != torch.float32:
        raise TypeError("weight gradients are fp32")
    wsp, wsn = (None, 0) if ws is None else (_ptr(ws), ws.numel())
    check(_lib.load().foremoe_grouped_ffn_wgrad(_ptr(x_perm), _ptr(h), _ptr(dy_perm), _ptr(d_au), _dt(x_perm),
                                                d, F, S, _ptr(slot_offset), _ptr(slot_gidx), G, n_cap,
                                                _ptr(dw_gate_up), _ptr(dw_down), wsp, wsn, _stream(x_perm.device)),
          "foremoe_grouped_ffn_wgrad")


def wgrad_steps(steps, *, a: str, b: str):
    """ctypes array of foremoe_wgrad_step records for the micro-steps in
    ``steps`` (mappings with tensors ``a`` and ``b`` named by the arguments,
    ``slot_offset``, ``slot_gidx``)."""
    arr = (_lib.WgradStep * max(len(steps), 1))()
    for i, st in enumerate(steps):
        A, B = st[a], st[b]
        arr[i] = _lib.WgradStep(_ptr(A), _ptr(B), _ptr(st["slot_offset"]), _ptr(st["slot_gidx"]),
                                int(st["slot_gidx"].shape[0]), int(A.shape[0]))
    return arr


def grouped_ffn_wgrad_steps(steps, dw_gate_up: torch.Tensor, dw_down: torch.Tensor,
                            ws: Optional[torch.Tensor] = None, part: int = 0, parts: int = 1) -> None:
    """Weight gradients of several micro-steps in one launch pair: each entry
    of ``steps`` maps x_perm, h, dy_perm, d_au, slot_offset, slot_gidx to that
    micro-step's tensors. Accumulates (+=) into dw_gate_up [G, 2F, d] and
    dw_down [G, d, F] (fp32); the same sum as one grouped_ffn_wgrad call per
    micro-step, in one read-modify-write of the gradients. ``part`` of
    ``parts``: only that share of the output tiles (all parts together give
    the whole update)."""
    G, F2, d = dw_gate_up.shape
    F = F2 // 2
    if dw_gate_up.dtype != torch.float32 or dw_down.dtype != torch.float32:
        raise TypeError("weight gradients are fp32")
    if not steps:
        return
    dt = _dt(steps[0]["x_perm"])
    wsp, wsn = (None, 0) if ws is None else (_ptr(ws), ws.numel())
    lib, st = _lib.load(), _stream(dw_gate_up.device)
    gu = wgrad_steps(steps, a="d_au", b="x_perm")
    check(lib.foremoe_ffn_gate_up_wgrad_steps(gu, len(steps), dt, d, F, G, part, parts, _ptr(dw_gate_up), wsp, wsn,
                                              st), "foremoe_ffn_gate_up_wgrad_steps")
    dn = wgrad_steps(steps, a="dy_perm", b="h")
    check(lib.foremoe_ffn_down_wgrad_steps(dn, len(steps), dt, d, F, G, part, parts, _ptr(dw_down), wsp, wsn, st),
          "foremoe_ffn_down_wgrad_steps")


def combine(y_perm: torch.Tensor, pair_to_row: torch.Tensor, gates: torch.Tensor,
            out_dtype: torch.dtype = torch.float32) -> torch.Tensor:
    T, K = gates.shape
    n_cap, d = y_perm.shape
    y = torch.empty((T, d), dtype=out_dtype, device=y_perm.device)
    check(_lib.load().foremoe_combine(_ptr(y_perm), _dt(y_perm), _ptr(pair_to_row), _ptr(gates), T, K, d, n_cap,
                                      y.data_ptr(), _DT[out_dtype], _stream(y_perm.device)), "foremoe_combine")
    return y


def combine_bwd(dy: torch.Tensor, y_perm: torch.Tensor, pair_to_row: torch.Tensor, gates: torch.Tensor,
                want_dgates: bool = True):
    T, K = gates.shape
    n_cap, d = y_perm.shape
    dy_perm = torch.empty((n_cap, d), dtype=dy.dtype, device=dy.device)
    dgates = torch.empty((T, K), dtype=torch.float32, device=dy.device) if want_dgates else None
    check(_lib.load().foremoe_combine_bwd(_ptr(dy), _ptr(y_perm), _dt(dy), _ptr(pair_to_row), _ptr(gates), T, K,
                                          d, n_cap, dy_perm.data_ptr(),
                                          None if dgates is None else dgates.data_ptr(), _stream(dy.device)),
          "foremoe_combine_bwd")
    return dy_perm, dgates


def permute_bwd(dx_perm: torch.Tensor, pair_to_row: torch.Tensor, T: int, K: int,
                out_dtype: torch.dtype = torch.float32) -> torch.Tensor:
    n_cap, d = dx_perm.shape
    dx = torch.empty((T, d), dtype=out_dtype, device=dx_perm.device)
    check(_lib.load().foremoe_permute_bwd(_ptr(dx_perm), _dt(dx_perm), _ptr(pair_to_row), T, K, d, n_cap,
                                          dx.data_ptr(), _DT[out_dtype], _stream(dx_perm.device)),
          "foremoe_permute_bwd")
    return dx


# ---------------------------------------------------------------------------
# Expert Transfer Engine, the part one GPU runs (see include/foremoe.h)
# ---------------------------------------------------------------------------
def xfer_record_bytes(d: int, F: int, dtype: torch.dtype, what: int) -> int:
    return int(_lib.load().foremoe_xfer_record_bytes(d, F, _DT[dtype], what))


def _host_list(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32).reshape(-1))


def copy_out(w_gate_up: torch.Tensor, w_down: torch.Tensor, dw_gate_up: torch.Tensor, dw_down: torch.Tensor,
             widx, gidx, what: int, buf: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Copy-out: records of weight slots widx / gradient slots gidx (host
    lists) packed into a send buffer (uint8 device tensor)."""
    W, F2, d = w_gate_up.shape
    F = F2 // 2
    G = dw_gate_up.shape[0]
    wi, gi = _host_list(widx), _host_list(gidx)
    n = len(wi)
    rb = xfer_record_bytes(d, F, w_gate_up.dtype, what)
    if buf is None:
        buf = torch.empty(n * rb, dtype=torch.uint8, device=w_gate_up.device)
    check(_lib.load().foremoe_copy_out(_ptr(w_gate_up), _ptr(w_down), _dt(w_gate_up), W, _ptr(dw_gate_up),
                                       _ptr(dw_down), G, d, F, n, wi.ctypes.data, gi.ctypes.data, what, _ptr(buf),
                                       buf.numel(), _stream(w_gate_up.device)), "foremoe_copy_out")
    return buf


def copy_in(buf: torch.Tensor, widx, gidx, gmode, what: int, w_gate_up: torch.Tensor, w_down: torch.Tensor,
            dw_gate_up: torch.Tensor, dw_down: torch.Tensor) -> None:
    """Copy-in: unpack the records of a receive buffer in place into the
    expert arrays (host lists widx, gidx, gmode)."""
    W, F2, d = w_gate_up.shape
    F = F2 // 2
    G = dw_gate_up.shape[0]
    wi, gi, gm = _host_list(widx), _host_list(gidx), _host_list(gmode)
    check(_lib.load().foremoe_copy_in(_ptr(buf), buf.numel(), len(wi), wi.ctypes.data, gi.ctypes.data,
                                      gm.ctypes.data, what, _ptr(w_gate_up), _ptr(w_down), _dt(w_gate_up), W,
                                      _ptr(dw_gate_up), _ptr(dw_down), G, d, F, _stream(buf.device)),
          "foremoe_copy_in")


def plan_prefetch(resident, needed):
    """(slot_of [n], fetch_expert [m], fetch_widx [m]) from the host planner."""
    res, need = _host_list(resident), _host_list(needed)
    n = len(need)
    slot_of = np.empty(max(n, 1), dtype=np.int32)
    fe = np.empty(max(n, 1), dtype=np.int32)
    fw = np.empty(max(n, 1), dtype=np.int32)
    nf = ctypes.c_int32(0)
    check(_lib.load().foremoe_plan_prefetch(res.ctypes.data, len(res), need.ctypes.data, n, slot_of.ctypes.data,
                                            fe.ctypes.data, fw.ctypes.data, ctypes.byref(nf)),
          "foremoe_plan_prefetch")
    return slot_of[:n].copy(), fe[:nf.value].copy(), fw[:nf.value].copy()


def prefetch_experts(host_gate_up: torch.Tensor, host_down: torch.Tensor, expert, widx, w_gate_up: torch.Tensor,
                     w_down: torch.Tensor, stream: Optional[torch.cuda.Stream] = None) -> None:
    """Host-to-device copies of experts from the pinned host master copy into
    weight slots, queued on ``stream`` (default: the current stream)."""
    if host_gate_up.is_cuda or host_down.is_cuda:
        raise ValueError("the master copy lives in host memory")
    E, F2, d = host_gate_up.shape
    W = w_gate_up.shape[0]
    ex, wi = _host_list(expert), _host_list(widx)
    st = (stream or torch.cuda.current_stream(w_gate_up.device)).cuda_stream
    check(_lib.load().foremoe_prefetch_experts(host_gate_up.data_ptr(), host_down.data_ptr(), E, _dt(host_gate_up),
                                               d, F2 // 2, len(ex), ex.ctypes.data, wi.ctypes.data, _ptr(w_gate_up),
                                               _ptr(w_down), W, st), "foremoe_prefetch_experts")


# ---------------------------------------------------------------------------
# Placement planner (host arrays; see include/foremoe.h)
# ---------------------------------------------------------------------------
def _machine(M: int, R: int, N_b: int, N_r: int) -> _lib.Machine:
    return _lib.Machine(int(M), int(R), int(N_b), int(N_r))


def _host_i32(a, shape=None) -> np.ndarray:
    out = np.ascontiguousarray(a, dtype=np.int32)
    if shape is not None and out.shape != tuple(shape):
        raise ValueError(f"expected shape {tuple(shape)}, got {out.shape}")
    return out


def plan_base(w_agg: np.ndarray, M: int, R: int, N_b: int, c_load: int = 1, c_traffic: int = 0) -> np.ndarray:
    """Stage 1: base rank [E] of every expert from the aggregate load [P, E]."""
    w = _host_i32(w_agg)
    P, E = w.shape
    if P != M * R:
        raise ValueError("w_agg must have M * R rows")
    out = np.empty(E, dtype=np.int32)
    mc = _machine(M, R, N_b, 0)
    check(_lib.load().foremoe_plan_base(w.ctypes.data, E, ctypes.byref(mc), int(c_load), int(c_traffic),
                                        out.ctypes.data), "foremoe_plan_base")
    return out


def plan_micro_step(w: np.ndarray, base_rank: np.ndarray, M: int, R: int, N_b: int, N_r: int, C_max: int):
    """Stages 2-4 of one micro-step: (copy_rank [E, C_max], counts [P, E, C_max], rank_load [P])."""
    w = _host_i32(w)
    P, E = w.shape
    if P != M * R:
        raise ValueError("w must have M * R rows")
    base = _host_i32(base_rank, (E,))
    copy_rank = np.empty((E, C_max), dtype=np.int32)
    counts = np.empty((P, E, C_max), dtype=np.int32)
    rank_load = np.empty(P, dtype=np.int64)
    mc = _machine(M, R, N_b, N_r)
    check(_lib.load().foremoe_plan_micro_step(w.ctypes.data, E, ctypes.byref(mc), base.ctypes.data, int(C_max),
                                              copy_rank.ctypes.data, counts.ctypes.data, rank_load.ctypes.data),
          "foremoe_plan_micro_step")
    return copy_rank, counts, rank_load


def plan_rank_slots(copy_rank: np.ndarray, rank: int, max_slots: int = _lib.MAX_SLOTS) -> dict:
    """One rank's slot table from a micro-step plan (host arrays)."""
    cr = _host_i32(copy_rank)
    E, C_max = cr.shape
    se = np.empty(max_slots, dtype=np.int32)
    sr = np.empty(max_slots, dtype=np.int32)
    sw = np.empty(max_slots, dtype=np.int32)
    nrep = np.empty(E, dtype=np.int32)
    local = np.empty(E, dtype=np.int32)
    S = ctypes.c_int32(0)
    W = ctypes.c_int32(0)
    check(_lib.load().foremoe_plan_rank_slots(cr.ctypes.data, E, C_max, int(rank), int(max_slots), se.ctypes.data,
                                              sr.ctypes.data, sw.ctypes.data, nrep.ctypes.data, local.ctypes.data,
                                              ctypes.byref(S), ctypes.byref(W)), "foremoe_plan_rank_slots")
    return dict(slot_expert=se[:S.value].copy(), slot_replica=sr[:S.value].copy(), slot_widx=sw[:S.value].copy(),
                expert_nrep=nrep, local_experts=local[:W.value].copy())
