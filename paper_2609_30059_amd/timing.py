"""Timing-only HIP events for the measurement tools (bench.py, the block gate,
the epilogue placement study).

A default HIP event performs a system-scope release when it is recorded: a
writeback and invalidation of the caches that costs the GPU about 3 us per
event and lengthens whatever interval it closes.  The events here are
created with hipEventDisableSystemFence, documented by HIP for events that
are used only to measure time; one costs about 1 us.  The HIP runtime is the
one torch has already loaded (looked up, never loaded anew), so torch's
streams are valid handles for it.
"""
from __future__ import annotations

import ctypes
import os

_HIP = None
DISABLE_SYSTEM_FENCE = 0x20000000


def _hip():
    global _HIP
    if _HIP is None:
        import torch  # noqa: F401  (loads the HIP runtime)
        hip = ctypes.CDLL("libamdhip64.so.7", mode=os.RTLD_NOLOAD)
        hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                            ctypes.c_void_p]
        hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        _HIP = hip
    return _HIP


class TimingEvent:
    """A HIP event used only for timing, recorded on torch's current stream;
    its timestamps are read only after a device synchronisation.  The same
    three calls as ``torch.cuda.Event(enable_timing=True)``."""

    def __init__(self):
        hip = _hip()
        self.ev = ctypes.c_void_p()
        rc = hip.hipEventCreateWithFlags(ctypes.byref(self.ev), DISABLE_SYSTEM_FENCE)
        if rc != 0:
            raise RuntimeError(f"hipEventCreateWithFlags failed ({rc})")

    def record(self):
        import torch
        rc = _hip().hipEventRecord(self.ev, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed ({rc})")

    def elapsed_time(self, end: "TimingEvent") -> float:
        """Milliseconds from this event to ``end``."""
        ms = ctypes.c_float()
        rc = _hip().hipEventElapsedTime(ctypes.byref(ms), self.ev, end.ev)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return ms.value

    def __del__(self):
        if _HIP is not None and getattr(self, "ev", None):
            _HIP.hipEventDestroy(self.ev)
