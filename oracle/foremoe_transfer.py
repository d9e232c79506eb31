"""Plain CPU oracle of the one-GPU half of ForeMoE's Expert Transfer Engine
(Sec. 6.1 CPU-assisted path; Sec. 6.2 per-layer transfer: Copy-out and
Copy-in; App. A.2 and A.3).

TEST INFRASTRUCTURE. Only tests/, the smoke check and the benchmark's CPU
baseline may import or run this module; the product path never does.

What it computes:

* ``copy_out`` - Copy-out (Sec. 6.2): the parameters and gradients of the
  experts leaving this GPU packed into one contiguous send buffer, one record
  per expert. A record holds the expert's parameters S_e = 3*h*h_ff*p_w
  bytes and/or its gradient S_g = 3*h*h_ff*p_g bytes (App. A.3), here in the
  order: gate/up parameters [2F, d], down parameters [d, F], gate/up
  gradient [2F, d], down gradient [d, F] (row-major, the weights' own
  layouts), p_g = 4 (App. A.4: fp32 gradient accumulation).
* ``copy_in`` - Copy-in (Sec. 6.2): the records of a receive buffer unpacked
  into the expert memory of this GPU. Parameters are copied into their
  weight slot. A gradient record either moves an expert's gradient here
  (``ASSIGN``: the target takes the record) or is a replica's partial
  gradient that is accumulated into the main expert's gradient (``ADD``:
  the target gains the record). Records naming the same target are applied
  in record order, starting from the target's current value, each step
  rounded to fp32 (the precision App. A.4 fixes), so the result is exact
  and unique.
* ``plan_prefetch`` - the CPU-assisted path (Sec. 6.1): of the experts the
  next micro-step needs, those not already resident in a weight slot are
  fetched from the host master copy into slots whose expert is not needed;
  resident ones stay where they are.

Readings where the paper is silent (listed in the design notes as well):
* record layout and order of the four parts (above); record i of a buffer
  starts at i times the record size;
* several records naming one gradient target are applied in record order;
* prefetch fills the free slots in ascending slot order with the missing
  experts in the order they are listed as needed.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np

PARAMS = 1
GRADS = 2
ASSIGN = 0
ADD = 1


def record_bytes(d: int, F: int, p_w: int, what: int) -> int:
    """Bytes of one record: S_e = 3*d*F*p_w with parameters, S_g = 3*d*F*4
    with gradients (App. A.3)."""
    n = 0
    if what & PARAMS:
        n += 3 * d * F * p_w
    if what & GRADS:
        n += 3 * d * F * 4
    return n


def _raw(a: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(a).reshape(-1).view(np.uint8)


def copy_out(w_gate_up: np.ndarray, w_down: np.ndarray, dw_gate_up: np.ndarray, dw_down: np.ndarray,
             widx: Sequence[int], gidx: Sequence[int], what: int) -> np.ndarray:
    """Send buffer (uint8) of len(widx) records: record i holds the parameters
    of weight slot widx[i] and/or the gradient of gradient slot gidx[i].

    w_gate_up [W, 2F, d], w_down [W, d, F] hold the parameters in their
    storage type (uint16 bf16 bit patterns, or float32); dw_gate_up
    [G, 2F, d], dw_down [G, d, F] are float32."""
    parts: List[np.ndarray] = []
    for i in range(len(widx)):
        if what & PARAMS:
            parts.append(_raw(w_gate_up[widx[i]]))
            parts.append(_raw(w_down[widx[i]]))
        if what & GRADS:
            parts.append(_raw(np.asarray(dw_gate_up[gidx[i]], dtype=np.float32)))
            parts.append(_raw(np.asarray(dw_down[gidx[i]], dtype=np.float32)))
    if not parts:
        return np.zeros(0, dtype=np.uint8)
    return np.concatenate(parts)


def copy_in(buf: np.ndarray, widx: Sequence[int], gidx: Sequence[int], gmode: Sequence[int], what: int,
            w_gate_up: np.ndarray, w_down: np.ndarray, dw_gate_up: np.ndarray,
            dw_down: np.ndarray) -> Tuple[np.ndarray, np.ndarray, np.ndarray, np.ndarray]:
    """Unpack a receive buffer of len(widx) records into copies of the four
    arrays and return them. widx[i] < 0 skips record i's parameters,
    gidx[i] < 0 its gradient."""
    W, F2, d = w_gate_up.shape
    F = F2 // 2
    p_w = w_gate_up.dtype.itemsize
    rb = record_bytes(d, F, p_w, what)
    wgu, wdn = w_gate_up.copy(), w_down.copy()
    ggu, gdn = dw_gate_up.astype(np.float32).copy(), dw_down.astype(np.float32).copy()
    buf = np.ascontiguousarray(buf, dtype=np.uint8)
    n_gu, n_dn = 2 * F * d, d * F
    for i in range(len(widx)):
        off = i * rb
        if what & PARAMS:
            a = buf[off:off + n_gu * p_w].view(w_gate_up.dtype).reshape(2 * F, d)
            off += n_gu * p_w
            b = buf[off:off + n_dn * p_w].view(w_down.dtype).reshape(d, F)
            off += n_dn * p_w
            if widx[i] >= 0:
                wgu[widx[i]] = a
                wdn[widx[i]] = b
        if what & GRADS:
            a = buf[off:off + n_gu * 4].view(np.float32).reshape(2 * F, d)
            off += n_gu * 4
            b = buf[off:off + n_dn * 4].view(np.float32).reshape(d, F)
            g = gidx[i]
            if g >= 0:
                if gmode[i] == ASSIGN:
                    ggu[g] = a
                    gdn[g] = b
                else:  # float32 + float32 -> float32, rounded to nearest (IEEE)
                    ggu[g] = ggu[g] + a
                    gdn[g] = gdn[g] + b
    return wgu, wdn, ggu, gdn


def plan_prefetch(resident: Sequence[int], needed: Sequence[int]) -> Tuple[List[int], List[Tuple[int, int]]]:
    """Weight slot of every needed expert, and the (expert, slot) fetches.

    resident[w] is the expert in weight slot w (-1: empty). Needed experts
    already resident keep their slot; each missing one, in the order listed,
    takes the lowest slot whose expert is not needed. Returns (slot_of
    [len(needed)], fetches)."""
    needed = [int(e) for e in needed]
    if len(set(needed)) != len(needed):
        raise ValueError("an expert is listed twice")
    where = {}
    for w, e in enumerate(resident):
        if e >= 0 and e not in where:
            where[int(e)] = w
    keep = {e for e in needed if e in where}
    free = [w for w, e in enumerate(resident) if not (e >= 0 and e in keep and where[int(e)] == w)]
    slot_of, fetches = [], []
    for e in needed:
        if e in keep:
            slot_of.append(where[e])
        else:
            if not free:
                raise ValueError("more experts needed than weight slots")
            w = free.pop(0)
            slot_of.append(w)
            fetches.append((e, w))
    return slot_of, fetches
