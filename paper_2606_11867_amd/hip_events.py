"""Device events for ordering and timing the micro-step schedule's streams.

torch's events complete with a system-scope release fence (so that the host
and peer devices see every earlier write). Ordering two streams of one GPU,
or timing a kernel, needs only the device-scope ordering that every
completion signal already gives, and the system fence costs time on the
stream that records: on MI355X, an event record between two kernels adds
about 2.9 us to that stream (1.0 us without the fence), a record that
another stream waits on 5.3 us (2.9 us), and a pair of timing events
attached to a kernel launch 7.0 us (3.1 us). These events are created with
hipEventDisableSystemFence. Results that the host reads are still made
visible by a device or stream synchronisation, which fences on its own.

The handles come from the HIP runtime that torch loaded (the library and
torch share it), so they can be passed to torch's streams and to the C ABI's
timed calls alike.
"""
from __future__ import annotations

import ctypes

_DISABLE_TIMING = 0x2
_DISABLE_SYSTEM_FENCE = 0x20000000

_rt = None


def _runtime():
    global _rt
    if _rt is None:
        import torch  # noqa: F401  (loads the HIP runtime; dlopen by soname then finds that copy)
        rt = ctypes.CDLL("libamdhip64.so.7")
        vp = ctypes.c_void_p
        rt.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(vp), ctypes.c_uint]
        rt.hipEventRecord.argtypes = [vp, vp]
        rt.hipStreamWaitEvent.argtypes = [vp, vp, ctypes.c_uint]
        rt.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), vp, vp]
        rt.hipEventSynchronize.argtypes = [vp]
        rt.hipEventDestroy.argtypes = [vp]
        for f in ("hipEventCreateWithFlags", "hipEventRecord", "hipStreamWaitEvent", "hipEventElapsedTime",
                  "hipEventSynchronize", "hipEventDestroy"):
            getattr(rt, f).restype = ctypes.c_int
        _rt = rt
    return _rt


def _check(rc: int, what: str) -> None:
    if rc != 0:
        raise RuntimeError(f"{what} failed with HIP error {rc}")


class Event:
    """A HIP event without the system-scope fence. timing=False also
    disables its timestamp (the cheapest form, for stream ordering only).
    Streams are torch streams (anything with a cuda_stream handle)."""

    def __init__(self, timing: bool = False):
        self._rt = _runtime()
        h = ctypes.c_void_p()
        flags = _DISABLE_SYSTEM_FENCE | (0 if timing else _DISABLE_TIMING)
        _check(self._rt.hipEventCreateWithFlags(ctypes.byref(h), flags), "hipEventCreateWithFlags")
        self.handle = h.value
        self.timing = timing

    # the name torch's events use for their handle, so that either kind can
    # be handed to the C ABI's timed calls
    @property
    def cuda_event(self) -> int:
        return self.handle

    def record(self, stream) -> None:
        _check(self._rt.hipEventRecord(self.handle, stream.cuda_stream), "hipEventRecord")

    def wait(self, stream) -> None:
        """Work queued on stream after this call waits for the event's last
        record."""
        _check(self._rt.hipStreamWaitEvent(stream.cuda_stream, self.handle, 0), "hipStreamWaitEvent")

    def synchronize(self) -> None:
        _check(self._rt.hipEventSynchronize(self.handle), "hipEventSynchronize")

    def elapsed_time(self, end: "Event") -> float:
        """Milliseconds from this event to end (both timing events, both
        completed)."""
        ms = ctypes.c_float()
        _check(self._rt.hipEventElapsedTime(ctypes.byref(ms), self.handle, end.handle), "hipEventElapsedTime")
        return float(ms.value)

    def __del__(self):
        h, self.handle = getattr(self, "handle", None), None
        if h and _rt is not None:
            _rt.hipEventDestroy(h)
