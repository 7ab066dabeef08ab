"""Binding of the vTime fair scheduler (``include/t2i_sched.h``): which
tenant's model-function invocation runs next on an idle executor (Sec. 6,
Alg. 1).  Argument marshalling only; the decisions are made in the library."""
from __future__ import annotations

import ctypes as C
from typing import Optional, Tuple

from . import _lib


class Scheduler:
    def __init__(self, delta: float):
        self.lib = _lib.load()
        h = C.c_void_p()
        _lib.check(self.lib.t2i_sched_create(float(delta), C.byref(h)))
        self.h = h

    def __del__(self):
        if getattr(self, "h", None):
            self.lib.t2i_sched_destroy(self.h)
            self.h = None

    def submit(self, tenant: int, fn_id: int, est: float, remaining: float, now: float):
        _lib.check(self.lib.t2i_sched_submit(self.h, tenant, fn_id, est, remaining, now))

    def schedule(self, now: float) -> Optional[Tuple[int, int, float]]:
        picked, fn, ten, ch = C.c_int32(), C.c_int64(), C.c_int32(), C.c_double()
        _lib.check(self.lib.t2i_sched_schedule(self.h, now, C.byref(picked), C.byref(fn),
                                               C.byref(ten), C.byref(ch)))
        return (fn.value, ten.value, ch.value) if picked.value else None

    def complete(self, fn_id: int, measured: float):
        _lib.check(self.lib.t2i_sched_complete(self.h, fn_id, measured))

    def vtime(self, tenant: int) -> float:
        v = C.c_double()
        _lib.check(self.lib.t2i_sched_vtime(self.h, tenant, C.byref(v)))
        return v.value
