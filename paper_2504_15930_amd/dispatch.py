"""ctypes binding of skewness-aware dispatching (``include/sl_dispatch.h``): marshalling only.

The algorithm (StreamRL Algorithm 2 with Equation 2) runs in ``libsl``'s C++;
this module converts numpy arrays and returns the plan.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import sl


class PtlProfile(ctypes.Structure):
    _fields_ = [("points", ctypes.c_int32), ("batch", ctypes.c_void_p), ("seconds", ctypes.c_void_p)]


_host_lib: ctypes.CDLL | None = None


def _lib():
    """libsl, or the host-only build of the dispatching code that the environment variable
    SL_DISPATCH_LIBRARY names (``build.build_dispatch_host``, e.g. with the host sanitizers)."""
    global _host_lib
    path = os.environ.get("SL_DISPATCH_LIBRARY")
    if path:
        if _host_lib is None:
            _host_lib = ctypes.CDLL(path)
        lib = _host_lib
    else:
        lib = sl.load()
    if not getattr(lib, "_dispatch_typed", False):
        P = ctypes.c_void_p
        lib.sl_generation_latency.argtypes = [ctypes.POINTER(PtlProfile), ctypes.c_double, ctypes.c_int32,
                                              ctypes.c_int32, ctypes.POINTER(ctypes.c_double)]
        lib.sl_dispatch_plan.argtypes = [P, ctypes.c_int32, ctypes.c_double, P, ctypes.c_int32, ctypes.c_int32,
                                         ctypes.POINTER(PtlProfile), ctypes.c_int32, ctypes.c_int32,
                                         ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32),
                                         ctypes.POINTER(ctypes.c_double), P]
        lib.sl_generation_latency.restype = ctypes.c_int
        lib.sl_dispatch_plan.restype = ctypes.c_int
        lib._dispatch_typed = True
    return lib


def _profile(batch, seconds):
    b = np.ascontiguousarray(batch, dtype=np.int32)
    s = np.ascontiguousarray(seconds, dtype=np.float64)
    if b.shape != s.shape or b.ndim != 1:
        raise ValueError("profile batch sizes and latencies must be 1-D and of equal length")
    return PtlProfile(len(b), b.ctypes.data, s.ctypes.data), (b, s)


def generation_latency(l_avg: float, m: int, max_batch: int, ptl_batch, ptl_seconds) -> float:
    """Equation 2 for one instance receiving ``m`` prompts."""
    prof, keep = _profile(ptl_batch, ptl_seconds)
    out = ctypes.c_double(0.0)
    sl._check(_lib().sl_generation_latency(ctypes.byref(prof), float(l_avg), int(m), int(max_batch),
                                           ctypes.byref(out)), "sl_generation_latency")
    return out.value


def plan(est_len, alpha: float, length_samples, num_instances: int, ptl_batch, ptl_seconds, max_batch: int,
         combine: str = "sum"):
    """Algorithm 2: returns (N_l, N_r, estimated latency, instance of every prompt)."""
    est = np.ascontiguousarray(est_len, dtype=np.int32)
    dist = np.ascontiguousarray(length_samples, dtype=np.int32)
    prof, keep = _profile(ptl_batch, ptl_seconds)
    inst = np.full(len(est), -1, dtype=np.int32)
    nl, nr, lat = ctypes.c_int32(0), ctypes.c_int32(0), ctypes.c_double(0.0)
    sl._check(_lib().sl_dispatch_plan(est.ctypes.data, len(est), float(alpha), dist.ctypes.data, len(dist),
                                      int(num_instances), ctypes.byref(prof), int(max_batch),
                                      1 if combine == "max" else 0, ctypes.byref(nl), ctypes.byref(nr),
                                      ctypes.byref(lat), inst.ctypes.data), "sl_dispatch_plan")
    return nl.value, nr.value, lat.value, inst
