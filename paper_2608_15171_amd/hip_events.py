"""hipEvent_t handles through the HIP runtime already loaded in the process.

The library's launches record such events when a call passes them (the
ppas_events argument of the planned calls), so a kernel's own duration can be
read on the stream it was launched on. Import after torch (the binding does), so the name
resolves to the runtime torch loaded.
"""
from __future__ import annotations

import ctypes


class HipEvents:
    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self) -> int:
        ev = ctypes.c_void_p()
        if self.hip.hipEventCreate(ctypes.byref(ev)) != 0:
            raise RuntimeError("hipEventCreate failed")
        return ev.value

    def elapsed_ms(self, start: int, stop: int) -> float:
        ms = ctypes.c_float()
        if self.hip.hipEventElapsedTime(ctypes.byref(ms), start, stop) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def destroy(self, ev: int) -> None:
        self.hip.hipEventDestroy(ev)
