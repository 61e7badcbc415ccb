"""Timing events for the benchmarks: HIP events of the process's own HIP
runtime (the one torch and libmec.so use), created with
hipEventDisableSystemFence. Recording such an event between two kernel
launches adds no system-scope acquire or release (no cache maintenance) to
the interval it measures; the timestamps are those of ordinary events.
"""
import ctypes


class HipEvent:
    """A timing event of the process's HIP runtime, created with
    hipEventDisableSystemFence (no system-scope acquire or release when it is
    recorded; the timestamps are the same)."""

    _rt = None
    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self):
        if HipEvent._rt is None:
            from . import _hip_runtimes
            paths = _hip_runtimes()
            if len(paths) != 1:
                raise RuntimeError("expected one HIP runtime in the process, found %r" % paths)
            rt = ctypes.CDLL(paths[0])
            rt.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            rt.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            rt.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                               ctypes.c_void_p]
            rt.hipEventDestroy.argtypes = [ctypes.c_void_p]
            HipEvent._rt = rt
        self.h = ctypes.c_void_p()
        self._check(HipEvent._rt.hipEventCreateWithFlags(ctypes.byref(self.h), self.DISABLE_SYSTEM_FENCE),
                    "hipEventCreateWithFlags")

    @staticmethod
    def _check(status, what):
        if status != 0:
            raise RuntimeError("%s failed with HIP status %d" % (what, status))

    def record(self, stream):
        self._check(HipEvent._rt.hipEventRecord(self.h, ctypes.c_void_p(stream.cuda_stream)),
                    "hipEventRecord")

    def elapsed_time(self, end):
        ms = ctypes.c_float()
        self._check(HipEvent._rt.hipEventElapsedTime(ctypes.byref(ms), self.h, end.h),
                    "hipEventElapsedTime")
        return ms.value

    def __del__(self):
        # at interpreter exit the class may already be torn down
        rt = getattr(HipEvent, "_rt", None) if HipEvent is not None else None
        if rt is not None and self.h:
            rt.hipEventDestroy(self.h)
