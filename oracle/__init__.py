"""CPU oracle of the global policy pass: TEST INFRASTRUCTURE ONLY.

A plain single-threaded C++ definition of the pass (``nalar_oracle.cpp``) and a
ctypes wrapper around it.  Only the test suite, ``__graft_entry__.smoke()`` and
the benchmark's ``cpu_baseline`` leg may import this package; the product path
(the HIP library and its binding) never does, and this package imports nothing
from the product.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading
from dataclasses import dataclass
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "nalar_oracle.cpp")
LIB = os.path.join(HERE, "libnalar_oracle.so")
CXXFLAGS = ["-O2", "-std=c++17", "-shared", "-fPIC", "-Wall", "-Wextra"]

OK, EINVAL, ECYCLE, ERANGE = 0, -1, -2, -3

# policy variants (the same bits as the library's problem flags)
POLICY_LPT = 2        # order by remaining critical path, longest first
POLICY_STATEFUL = 4   # a future whose state lives on an instance of its type runs there
POLICY_GREEDY = 8     # route in output order, each future adding its service time to its instance
POLICY_SRTF = 16      # order by remaining critical path, shortest first
POLICY_WEIGHTED = 32  # deal each type's futures to its instances by weight, in output order

_lock = threading.Lock()
_lib: Optional[ctypes.CDLL] = None


def build(force: bool = False) -> str:
    """Compile the oracle with g++ (always when ``force``)."""
    with _lock:
        stale = (not os.path.exists(LIB)) or os.path.getmtime(LIB) < os.path.getmtime(SRC)
        if force or stale:
            tmp = LIB + ".tmp"
            subprocess.run(["g++", *CXXFLAGS, SRC, "-o", tmp], check=True)
            os.replace(tmp, LIB)
    return LIB


def _load() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(LIB)
        P = ctypes.c_void_p
        I64 = ctypes.c_int64
        lib.nalar_oracle_pass.restype = ctypes.c_int
        lib.nalar_oracle_pass.argtypes = [I64] * 6 + [P] * 17
        lib.nalar_oracle_pass_policy.restype = ctypes.c_int
        lib.nalar_oracle_pass_policy.argtypes = [I64] * 6 + [ctypes.c_uint32] + [P] * 19
        _lib = lib
    return _lib


@dataclass
class OracleResult:
    status: int
    n_ready: int
    rem: Optional[np.ndarray]
    order: np.ndarray
    slack: np.ndarray
    route: np.ndarray
    cost: np.ndarray


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def run(p, *, want_rem: bool = True, override: Optional[dict] = None,
        policy: int = 0, priority: Optional[np.ndarray] = None,
        weights: Optional[np.ndarray] = None) -> OracleResult:
    """Run the oracle on a problem (any object with the workloads.Problem
    fields).  ``override`` may replace scalar sizes or set arrays to None, to
    exercise validation; ``policy`` selects the variants (POLICY_* bits),
    ``priority`` (uint8 per workflow, or None) the priority levels and
    ``weights`` (uint32 per instance, or None) the weights of POLICY_WEIGHTED."""
    lib = _load()
    o = dict(N=p.n_nodes, E=p.n_edges, W=p.n_workflows, M=p.n_instances,
             now=p.now_us, mig=p.migration_cost_us)
    arrays = {f: np.ascontiguousarray(getattr(p, f)) for f in (
        "wf", "type", "est_us", "done", "loc", "dep_off", "dep_idx", "deadline_us",
        "inst_type", "inst_load_us", "inst_speed_permille")}
    if override:
        for k, v in override.items():
            if k in o:
                o[k] = v
            else:
                arrays[k] = v
    n_out = max(int(p.n_nodes), 1)
    rem = np.zeros(n_out, np.int64) if want_rem else None
    order = np.zeros(n_out, np.int32)
    slack = np.zeros(n_out, np.int64)
    route = np.zeros(n_out, np.int32)
    cost = np.zeros(n_out, np.int64)
    n_ready = ctypes.c_int64(0)
    prio = None if priority is None else np.ascontiguousarray(priority, dtype=np.uint8)
    wts = None if weights is None else np.ascontiguousarray(weights, dtype=np.uint32)
    rc = lib.nalar_oracle_pass_policy(
        o["N"], o["E"], o["W"], o["M"], o["now"], o["mig"], policy, _ptr(prio), _ptr(wts),
        *[_ptr(arrays[f]) for f in ("wf", "type", "est_us", "done", "loc", "dep_off",
                                    "dep_idx", "deadline_us", "inst_type", "inst_load_us",
                                    "inst_speed_permille")],
        _ptr(rem), _ptr(order), _ptr(slack), _ptr(route), _ptr(cost), ctypes.byref(n_ready))
    R = int(n_ready.value) if rc == OK else 0
    return OracleResult(rc, R, None if rem is None else rem[: p.n_nodes], order[:R],
                        slack[:R], route[:R], cost[:R])
