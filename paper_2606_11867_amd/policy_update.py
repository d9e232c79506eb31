"""One policy-update micro-step of the expert layer through the C ABI, in the
launch configuration the benchmark times (Sec. 7.1: the policy update runs
forward and backward per micro-step; Sec. 6.2 and App. A.4: the expert
gradients accumulate in fp32 over the micro-steps).

Only ABI calls and stream ordering live here; every step of the path runs in
libforemoe.so. A micro-step is

  histogram + assign_replicas (one call) -> permute -> gate/up (+SwiGLU) -> down
  -> combine -> combine_bwd -> down dgrad (+SwiGLU') -> gate/up dgrad
  -> gate/up wgrad, down wgrad -> permute_bwd

Schedules:
  * one stream: every call in that order;
  * overlap: the two weight-gradient GEMMs run on a second stream (default
    priority), each beside the data-gradient GEMM that does not feed it
    (down wgrad beside down dgrad, gate/up wgrad beside gate/up dgrad); both
    share one workspace, so they stay ordered on that stream, and the main
    stream waits for it at the end of the micro-step;
  * pipelined: as overlap, but the streams are never joined: micro-step i
    uses activation buffer set i % 2 and, before reusing it, the main
    stream waits for the side-stream work of micro-step i - 2, so the next
    micro-step's dispatch and forward start while this one's weight
    gradients run;
  * side_gathers (with overlap): permute_bwd (1), and also the combine (2),
    move to the second stream, after the weight gradients; their outputs
    feed nothing later in the micro-step, so the main stream goes on to the
    next micro-step right after the gate/up dgrad. A caller reading dx (or
    y) waits for the second stream first.

Weight gradients grouped over micro-steps (wgrad_group M > 1): the two
weight-gradient GEMMs of a group of M consecutive micro-steps run as one
launch pair over all M micro-steps' rows (App. A.4: the fp32 expert
gradients accumulate over the micro-steps of an update step; one
read-modify-write of dW then serves M micro-steps), after the gate/up dgrad
of the group's last micro-step, on a third stream, while the next group's
micro-steps run. The operands they read (x_perm, h, dy_perm, d_au and the
slot offsets) live in a ring of 2M + 1 buffer sets; micro-step i rewrites
the set of micro-step i - 2M - 1 only after the launch that read it is done.
finish() launches the weight gradients of an incomplete last group.
Micro-step indices between start() and finish() must be consecutive, and
the schedule (pipelined or not) the same.
"""
from __future__ import annotations

import ctypes
from typing import Dict, List, Optional

import torch

from . import _lib
from .api import DevicePlan, ffn_workspace, wgrad_workspace, workspace
from .hip_events import Event

PHASES = ["histogram_assign", "permute", "gate_up_fwd", "down_fwd", "combine", "combine_bwd",
          "down_dgrad", "gate_up_dgrad", "gate_up_wgrad", "down_wgrad", "permute_bwd"]
# row-GEMM phases: one kernel each, timed by events attached to the launch
ROW_GEMMS = {"gate_up_fwd", "down_fwd", "down_dgrad", "gate_up_dgrad"}


class MicroStep:
    """The resident inputs of one micro-step: routing, gates, tokens, the
    upstream gradient and the slot table, all device tensors."""

    def __init__(self, ids: torch.Tensor, gates: torch.Tensor, x: torch.Tensor, dy: torch.Tensor,
                 plan: DevicePlan):
        self.ids, self.gates, self.x, self.dy, self.plan = ids, gates, x, dy, plan
        self.cplan = plan.c_struct()
        self.S = plan.S


class PolicyUpdate:
    """Buffers, workspaces and streams for running micro-steps of one rank's
    share (T tokens, top-K, width d, FFN width F, E experts, G gradient
    groups, at most S_max slots) with bf16 activations and weights, and the
    fp32 weight gradients dw_gate_up [G, 2F, d], dw_down [G, d, F] that every
    micro-step accumulates into.

    split: give the row GEMMs their workspace (a partial last round of tiles
    is cut along K). n_cap: rows of the permuted buffers (default T * K, every
    pair local; a rank share needs only its largest local pair count).
    wgrad_group: micro-steps per weight-gradient launch pair (1: every
    micro-step its own, beside its data-gradient GEMMs; the benchmark uses
    8: ring of 17 sets of x_perm, h, dy_perm, d_au)."""

    def __init__(self, T: int, K: int, d: int, F: int, E: int, G: int, S_max: int, w_gate_up: torch.Tensor,
                 w_down: torch.Tensor, device, split: bool = True, y_dtype=torch.bfloat16,
                 dx_dtype=torch.bfloat16, n_cap: Optional[int] = None, wgrad_group: int = 1):
        self.lib = _lib.load()
        self.T, self.K, self.d, self.F, self.E, self.G = T, K, d, F, E, G
        M = int(wgrad_group)
        if not 1 <= M <= _lib.MAX_WGRAD_STEPS or M * S_max > _lib.MAX_SLOTS:
            raise ValueError(f"wgrad_group={M}: 1..{_lib.MAX_WGRAD_STEPS} micro-steps of at most "
                             f"{_lib.MAX_SLOTS} slots in all")
        self.M = M
        self.R = 2 * M + 1 if M > 1 else 2  # weight-gradient operand sets
        self.dev = torch.device(device)
        self.n_cap = T * K if n_cap is None else int(n_cap)
        self.gu, self.dn = w_gate_up, w_down
        self.y_dt, self.dx_dt = _lib.BF16 if y_dtype == torch.bfloat16 else _lib.F32, \
            _lib.BF16 if dx_dtype == torch.bfloat16 else _lib.F32
        bf = torch.bfloat16
        dev = self.dev
        z = lambda *s, dt=bf: torch.zeros(s, dtype=dt, device=dev)  # noqa: E731
        n_cap = self.n_cap

        def buffer_set():
            return dict(
                counts=z(E, dt=torch.int32), rep_begin=z(E, 17, dt=torch.int32), slot_count=z(S_max, dt=torch.int32),
                ws=workspace(T, K, E, dev), r2p=z(n_cap, dt=torch.int32), p2r=z(T * K, dt=torch.int32),
                y_perm=z(n_cap, d), au=z(n_cap, 2 * F), y=z(T, d, dt=y_dtype), dgates=z(T, K, dt=torch.float32),
                dx_perm=z(n_cap, d), dx=z(T, d, dt=dx_dtype))

        def wgrad_set():  # what the weight gradients read
            return dict(slot_offset=z(S_max + 1, dt=torch.int32), x_perm=z(n_cap, d), h=z(n_cap, F),
                        dy_perm=z(n_cap, d), d_au=z(n_cap, 2 * F))

        # two activation sets: the next micro-step's forward can start while
        # this one's weight gradients (or second-stream gathers) still read
        # its set; the weight-gradient operands in a ring of R sets
        self.sets: List[Dict[str, torch.Tensor]] = [buffer_set(), buffer_set()]
        self.wsets: List[Dict[str, torch.Tensor]] = [wgrad_set() for _ in range(self.R)]
        self.dw_gate_up = z(G, 2 * F, d, dt=torch.float32)
        self.dw_down = z(G, d, F, dt=torch.float32)
        self.wws = wgrad_workspace(d, F, dev)
        self.rws = ffn_workspace(dev) if split else None
        self.main = torch.cuda.current_stream(dev)
        self.side = torch.cuda.Stream(dev)  # default priority, like every stream here
        # grouped weight gradients run on a third stream; gdone[k % 4]: group
        # k's launch pair is done
        self.wside = torch.cuda.Stream(dev) if M > 1 else None
        self.gdone = [Event() for _ in range(4)]
        # stream ordering uses events without the system-scope fence (both
        # streams are on this GPU; the fence would cost the recording stream
        # a few microseconds per record)
        self.done = [Event(), Event()]  # side-stream work of the micro-step using set b
        # early_hist: the histogram + replica split of the micro-step using
        # set b, run on the second stream during the micro-step before it
        self.hdone = [Event(), Event()]
        # micro-step index -> (inputs, activation set, weight-gradient set)
        # its early launch used
        self._early: Dict[int, tuple] = {}
        self._dep = [Event() for _ in range(8)]  # the cross-stream dependencies of one micro-step
        self._join = Event()
        self._ptrs = [{k: v.data_ptr() for k, v in st.items()} for st in self.sets]
        self._wptrs = [{k: v.data_ptr() for k, v in st.items()} for st in self.wsets]
        self.wmeta: List[Optional[MicroStep]] = [None] * self.R  # the micro-step whose operands a set holds
        self._pipelined = False  # the schedule of the micro-steps run since start() / finish()
        self._first: Optional[int] = None  # first and last micro-step run since start() / finish()
        self._last: Optional[int] = None
        self._flush_stream = self.main

    def _indices(self, i: int, pipelined: bool):
        b = i % 2 if pipelined else 0
        wb = i % self.R if (pipelined or self.M > 1) else 0
        return b, wb

    def set_of(self, i: int, pipelined: bool) -> Dict[str, torch.Tensor]:
        """The activation buffers micro-step i uses under that schedule."""
        b, wb = self._indices(i, pipelined)
        return {**self.sets[b], **self.wsets[wb]}

    def wgrad_launches_at(self, i: int) -> bool:
        """Whether micro-step i launches weight gradients (grouped: the last
        of its group; indices consecutive from a multiple of M)."""
        return i % self.M == self.M - 1

    def start(self) -> None:
        """Before the first pipelined micro-step: nothing to wait for yet, and
        no early launch of an earlier sequence is used (its sets may have
        been rewritten since)."""
        self._early.clear()
        for e in self.done + self.gdone:
            e.record(self.side)

    def _group(self, k: int, upto: Optional[int] = None) -> list:
        """(set, micro-step) of the micro-steps of group k run since start()
        (up to micro-step `upto`)."""
        M, R = self.M, self.R
        if self._first is None:
            return []
        hi = k * M + M - 1 if upto is None else min(upto, k * M + M - 1)
        return [(j % R, self.wmeta[j % R]) for j in range(max(k * M, self._first), hi + 1)]

    def finish(self, ev: Optional[dict] = None) -> bool:
        """Launch the weight gradients of an incomplete last group, then join
        the other streams into the main stream. ev: optional timing events of
        the two weight-gradient phases, around that launch. Returns whether
        there was such a launch."""
        flushed = False
        if self.M > 1 and self._last is not None and not self.wgrad_launches_at(self._last):
            flushed = True
            last = self._last
            members = self._group(last // self.M, last)
            st = self._flush_stream
            if st is not self.main:
                self._join.record(self.main)
                self._join.wait(st)
            for phase in ("down_wgrad", "gate_up_wgrad"):
                if ev is not None and phase in ev:
                    ev[phase][0].record(st)
                _lib.check(self._wgrad_call(phase, members, 0, 1)(st.cuda_stream), phase)
                if ev is not None and phase in ev:
                    ev[phase][1].record(st)
        self._first = self._last = None
        self._early.clear()
        for st in (self.side, self.wside):
            if st is not None:
                self._join.record(st)
                self._join.wait(self.main)
        return flushed

    def _wgrad_call(self, phase: str, members: list, part: int, parts: int):
        """The weight-gradient call of one phase over the micro-steps in
        members, output part `part` of `parts`, as a function of the stream."""
        lib, d, F, G = self.lib, self.d, self.F, self.G
        wws, wwsz = self.wws.data_ptr(), self.wws.numel()
        n = len(members)
        if phase == "gate_up_wgrad":
            a, b, fn, dw = "d_au", "x_perm", lib.foremoe_ffn_gate_up_wgrad_steps, self.dw_gate_up.data_ptr()
        else:
            a, b, fn, dw = "dy_perm", "h", lib.foremoe_ffn_down_wgrad_steps, self.dw_down.data_ptr()
        recs = (_lib.WgradStep * n)(*[_lib.WgradStep(self._wptrs[wb][a], self._wptrs[wb][b],
                                                     self._wptrs[wb]["slot_offset"], ms.plan.slot_gidx.data_ptr(),
                                                     ms.S, self.n_cap) for wb, ms in members])
        return lambda q: fn(recs, n, _lib.BF16, d, F, G, part, parts, dw, wws, wwsz, q)

    def ops(self, i: int, ms: MicroStep, ev: Optional[dict] = None, overlap: bool = False,
            pipelined: bool = False, side_gathers: int = 0, fwd_after_side: bool = False,
            next_ms: Optional[MicroStep] = None, early_hist: bool = False) -> list:
        """The operations of micro-step i on inputs ms, in order, as (phase,
        thunk) pairs (phase None: a stream dependency). ev maps phases to
        (begin, end) timing events (hip_events.Event or torch's): row GEMMs
        carry theirs on the kernel launch, the other phases are bracketed by event records on the stream
        the phase runs on. side_gathers (with overlap): 1 runs permute_bwd,
        2 also the combine, on the second stream (their outputs feed nothing
        later in the micro-step). early_hist (pipelined, with next_ms, the
        inputs of micro-step i + 1): micro-step i + 1's histogram + replica
        split runs on the second stream after this micro-step's down forward
        (beside its combine), and micro-step i + 1 starts with the permute;
        except after the last micro-step of a weight-gradient group. The
        returned operations must be run, in order (run() does): building
        them consumes the record of such an early launch."""
        lib, main, side = self.lib, self.main, self.side
        overlap = overlap or pipelined
        bset, wset = self._indices(i, pipelined)
        P = {**self._ptrs[bset], **self._wptrs[wset]}
        M = self.M
        T, K, d, F, G, n_cap = self.T, self.K, self.d, self.F, self.G, self.n_cap
        S = ms.S
        so = P["slot_offset"]
        widx, gidx = ms.plan.slot_widx.data_ptr(), ms.plan.slot_gidx.data_ptr()
        cp = ctypes.byref(ms.cplan)
        wsz = self.sets[bset]["ws"].numel()
        rws, rwsz = (None, 0) if self.rws is None else (self.rws.data_ptr(), self.rws.numel())
        wws, wwsz = self.wws.data_ptr(), self.wws.numel()
        gu, dn = self.gu.data_ptr(), self.dn.data_ptr()
        dwgu, dwdn = self.dw_gate_up.data_ptr(), self.dw_down.data_ptr()
        BF16 = _lib.BF16
        ops = []

        def call(phase, st, rc_fn):
            def run():
                timed = ev is not None and phase in ev
                if phase in ROW_GEMMS:
                    e = (ev[phase][0].cuda_event, ev[phase][1].cuda_event) if timed else (None, None)
                    _lib.check(rc_fn(st.cuda_stream, *e), phase)
                    return
                if timed:
                    ev[phase][0].record(st)
                _lib.check(rc_fn(st.cuda_stream), phase)
                if timed:
                    ev[phase][1].record(st)
            ops.append((phase, run))

        n_dep = [0]

        def dep(waiter, on):
            e = self._dep[n_dep[0]]  # its record and the wait for it are queued back to back
            n_dep[0] += 1

            def run():
                e.record(on)
                e.wait(waiter)
            ops.append((None, run))

        def gate_up_wgrad(st):
            call("gate_up_wgrad", st, lambda q: lib.foremoe_ffn_gate_up_wgrad(
                P["d_au"], P["x_perm"], BF16, d, F, S, so, gidx, G, n_cap, dwgu, wws, wwsz, q))

        def down_wgrad(st):
            call("down_wgrad", st, lambda q: lib.foremoe_ffn_down_wgrad(
                P["dy_perm"], P["h"], BF16, d, F, S, so, gidx, G, n_cap, dwdn, wws, wwsz, q))

        if pipelined:
            # set bset was last used two micro-steps ago: its second-stream
            # work (M = 1: its weight gradients too) must be done
            ops.append((None, lambda: self.done[bset].wait(main)))
        k = i // M
        if pipelined and M > 1 and i - self.R >= (self._first if self._first is not None else i):
            # set wset was last read by the launch pair of group (i - R) // M
            gq = ((i - self.R) // M) % 4
            ops.append((None, lambda: self.gdone[gq].wait(main)))
        early = pipelined and early_hist
        run_hist = True
        if i in self._early:  # launched during micro-step i - 1: its writes land first
            ems, eb, ewb = self._early.pop(i)
            ops.append((None, lambda: self.hdone[eb].wait(main)))
            # other inputs than announced, or other sets (another schedule): run it again
            run_hist = not (ems is ms and eb == bset and ewb == wset)
        if run_hist:
            call("histogram_assign", main, lambda q: lib.foremoe_histogram_assign(
                ms.ids.data_ptr(), T, K, cp, P["counts"], P["rep_begin"], P["slot_count"], so, P["ws"], wsz, q))
        call("permute", main, lambda q: lib.foremoe_permute(
            ms.x.data_ptr(), BF16, T, d, ms.ids.data_ptr(), K, cp, P["rep_begin"], so, n_cap, P["x_perm"],
            P["r2p"], P["p2r"], P["ws"], wsz, q))
        if pipelined and fwd_after_side:  # the previous micro-step's second-stream work ends first
            prev = self.done[(i - 1) % 2]
            ops.append((None, lambda: prev.wait(main)))
        call("gate_up_fwd", main, lambda q, e0, e1: lib.foremoe_ffn_gate_up_fwd_timed(
            P["x_perm"], BF16, d, F, S, so, widx, G, gu, n_cap, P["h"], P["au"], rws, rwsz, q, e0, e1))
        call("down_fwd", main, lambda q, e0, e1: lib.foremoe_ffn_down_fwd_timed(
            P["h"], BF16, d, F, S, so, widx, G, dn, n_cap, P["y_perm"], rws, rwsz, q, e0, e1))
        if early and next_ms is not None and not (M > 1 and self.wgrad_launches_at(i)):
            # (not after the last micro-step of a group: the group's weight-
            # gradient kernels, launched at its end, hold every CU for a while,
            # and the next micro-step's own histogram, on the main stream,
            # then takes that wait instead of its gate/up forward)
            # micro-step i + 1's sets: the activation set of micro-step i - 1,
            # whose main-stream kernels are done once this micro-step's have
            # started, and a weight-gradient set last read by the grouped
            # launch of micro-step i + 1 - R (M > 1)
            j = i + 1
            nb, nwb = self._indices(j, pipelined)
            NP = {**self._ptrs[nb], **self._wptrs[nwb]}
            dep(side, main)
            if M > 1 and j - self.R >= (self._first if self._first is not None else i):
                hq = ((j - self.R) // M) % 4
                ops.append((None, lambda: self.gdone[hq].wait(side)))
            ncp = ctypes.byref(next_ms.cplan)
            ops.append(("histogram_assign", lambda: _lib.check(lib.foremoe_histogram_assign(
                next_ms.ids.data_ptr(), T, K, ncp, NP["counts"], NP["rep_begin"], NP["slot_count"],
                NP["slot_offset"], NP["ws"], self.sets[nb]["ws"].numel(), side.cuda_stream), "histogram_assign")))
            ops.append((None, lambda: self.hdone[nb].record(side)))
            ops.append((None, lambda: self._early.__setitem__(j, (next_ms, nb, nwb))))
        if overlap and side_gathers >= 2:
            dep(side, main)
        call("combine", side if overlap and side_gathers >= 2 else main, lambda q: lib.foremoe_combine(
            P["y_perm"], BF16, P["p2r"], ms.gates.data_ptr(), T, K, d, n_cap, P["y"], self.y_dt, q))
        call("combine_bwd", main, lambda q: lib.foremoe_combine_bwd(
            ms.dy.data_ptr(), P["y_perm"], BF16, P["p2r"], ms.gates.data_ptr(), T, K, d, n_cap,
            P["dy_perm"], P["dgates"], q))
        if overlap and M == 1:
            dep(side, main)
            down_wgrad(side)
        call("down_dgrad", main, lambda q, e0, e1: lib.foremoe_ffn_down_dgrad_timed(
            P["dy_perm"], P["au"], BF16, d, F, S, so, widx, G, dn, n_cap, P["d_au"], rws, rwsz, q, e0, e1))
        if overlap and M == 1:
            dep(side, main)
            gate_up_wgrad(side)
        call("gate_up_dgrad", main, lambda q, e0, e1: lib.foremoe_ffn_gate_up_dgrad_timed(
            P["d_au"], BF16, d, F, S, so, widx, G, gu, n_cap, P["dx_perm"], rws, rwsz, q, e0, e1))
        if not overlap and M == 1:  # same order as on the side stream: down, then gate/up
            down_wgrad(main)
            gate_up_wgrad(main)
        if overlap and side_gathers >= 1:
            dep(side, main)
        call("permute_bwd", side if overlap and side_gathers >= 1 else main, lambda q: lib.foremoe_permute_bwd(
            P["dx_perm"], BF16, P["p2r"], T, K, d, n_cap, P["dx"], self.dx_dt, q))
        if pipelined:
            ops.append((None, lambda: self.done[bset].record(side)))
        if M > 1 and self.wgrad_launches_at(i):
            # the whole group in one launch pair, on a third stream when overlapped
            grp = self._group(k, i - 1) + [(wset, ms)] if self._first is not None else [(wset, ms)]
            wst = self.wside if overlap else main
            if overlap:
                dep(wst, main)
            for phase in ("down_wgrad", "gate_up_wgrad"):
                call(phase, wst, self._wgrad_call(phase, grp, 0, 1))
            if pipelined:
                ops.append((None, lambda: self.gdone[k % 4].record(wst)))
            elif overlap:
                dep(main, wst)
        if overlap and not pipelined:
            dep(main, side)
        return ops

    def run(self, i: int, ms: MicroStep, ev: Optional[dict] = None, overlap: bool = False,
            pipelined: bool = False, side_gathers: int = 0, fwd_after_side: bool = False,
            next_ms: Optional[MicroStep] = None, early_hist: bool = False) -> None:
        if self._first is not None and pipelined != self._pipelined:
            # the buffer sets and the waits that guard them depend on it
            raise ValueError("pipelined cannot change between start() and finish()")
        self._pipelined = pipelined
        ops = self.ops(i, ms, ev, overlap, pipelined, side_gathers, fwd_after_side, next_ms, early_hist)
        _, wset = self._indices(i, pipelined)
        self.wmeta[wset] = ms
        if self._first is None:
            self._first = i
        self._last = i
        self._flush_stream = self.wside if (overlap or pipelined) and self.M > 1 else self.main
        for _, op in ops:
            op()
