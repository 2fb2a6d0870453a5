"""Timing events from the HIP runtime (ctypes), for kernel tracing.

Uses the HIP runtime already loaded by torch (same soname as libflowmoe's),
so events, streams and the library share one runtime.
"""
from __future__ import annotations

import ctypes

_hip = None


def hip():
    global _hip
    if _hip is None:
        import torch  # noqa: F401  (loads the runtime first)
        lib = ctypes.CDLL("libamdhip64.so.7")
        lib.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        lib.hipEventCreate.restype = ctypes.c_int
        lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
        lib.hipEventDestroy.restype = ctypes.c_int
        lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                            ctypes.c_void_p]
        lib.hipEventElapsedTime.restype = ctypes.c_int
        lib.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        lib.hipEventSynchronize.restype = ctypes.c_int
        _hip = lib
    return _hip


class EventArray:
    """2 * pairs timing events in a ctypes array (begin/end pairs)."""

    def __init__(self, pairs: int):
        self.pairs = pairs
        self.ev = (ctypes.c_void_p * (2 * pairs))()
        self.kinds = (ctypes.c_int32 * max(pairs, 1))()
        h = hip()
        for i in range(2 * pairs):
            e = ctypes.c_void_p()
            rc = h.hipEventCreate(ctypes.byref(e))
            if rc != 0:
                raise RuntimeError(f"hipEventCreate failed ({rc})")
            self.ev[i] = e.value

    def elapsed_ms(self, i: int) -> float:
        """Milliseconds between the begin and end events of pair i."""
        h = hip()
        rc = h.hipEventSynchronize(self.ev[2 * i + 1])
        if rc != 0:
            raise RuntimeError(f"hipEventSynchronize failed ({rc})")
        out = ctypes.c_float()
        rc = h.hipEventElapsedTime(ctypes.byref(out), self.ev[2 * i], self.ev[2 * i + 1])
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return float(out.value)

    def close(self) -> None:
        h = hip()
        for i in range(2 * self.pairs):
            if self.ev[i]:
                h.hipEventDestroy(self.ev[i])
                self.ev[i] = None

    def __del__(self):  # pragma: no cover
        try:
            self.close()
        except Exception:
            pass
