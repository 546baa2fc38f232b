"""Events that order two streams of one device.

Created without timing and without the system-scope fence
(hipEventDisableSystemFence): recording one releases at device scope only,
which is all another stream of the same device needs; the host still waits
for work with a device or stream synchronisation.  The calls go to the HIP
runtime that torch has already loaded.  record(stream) / wait(stream) have
the meaning of torch.cuda.Event's methods of the same names.
"""
from __future__ import annotations


class StreamEvent:
    """One such event (see the module's description)."""
    _hip = None

    @classmethod
    def hip(cls):
        if cls._hip is None:
            import ctypes
            path = None
            with open("/proc/self/maps") as f:
                for line in f:
                    if "libamdhip64" in line:
                        path = line.split()[-1]
                        break
            if path is None:
                raise RuntimeError("the HIP runtime is not loaded")
            lib = ctypes.CDLL(path)
            lib.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            lib.hipStreamWaitEvent.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint]
            lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
            cls._hip = lib
        return cls._hip

    def __init__(self):
        import ctypes
        self.h = ctypes.c_void_p()
        rc = self.hip().hipEventCreateWithFlags(ctypes.byref(self.h), 0x2 | 0x20000000)
        if rc != 0:
            raise RuntimeError("hipEventCreateWithFlags failed (%d)" % rc)

    def record(self, stream):
        rc = self.hip().hipEventRecord(self.h, stream.cuda_stream)
        if rc != 0:
            raise RuntimeError("hipEventRecord failed (%d)" % rc)

    def wait(self, stream):
        """Make stream wait for the last record of this event."""
        rc = self.hip().hipStreamWaitEvent(stream.cuda_stream, self.h, 0)
        if rc != 0:
            raise RuntimeError("hipStreamWaitEvent failed (%d)" % rc)

    def __del__(self):
        if self._hip is not None and self.h:
            self._hip.hipEventDestroy(self.h)
