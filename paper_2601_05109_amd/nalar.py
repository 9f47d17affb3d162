"""ctypes binding of the C ABI in include/nalar_policy.h.

Argument marshalling only: every step of the pass runs in the HIP library
``libnalar_policy.so`` built from ``csrc/``.  Loading fails loudly when the
library is missing; there is no other implementation behind these names.

Functions with the C names (``nalar_policy_create``, ``nalar_policy_pass``,
``nalar_policy_destroy``, ``nalar_policy_last_error``, ``nalar_policy_set_timing``,
``nalar_policy_get_timing``) take and return the ctypes structures below.  The
``Policy`` class and ``DeviceProblem`` are conveniences over them for torch
device tensors.
"""
from __future__ import annotations

import atexit
import ctypes
import os
import sys
import weakref
from dataclasses import dataclass
from typing import Optional

_is_finalizing = sys.is_finalizing  # kept: sys may be cleared before late finalizers run

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libnalar_policy.so")

NALAR_OK, NALAR_EINVAL, NALAR_ECYCLE, NALAR_ERANGE, NALAR_ENOMEM, NALAR_EDEVICE = 0, -1, -2, -3, -4, -5
NALAR_WF_CONTIGUOUS = 1
NALAR_ORDER_LPT = 2          # problem flag: order by remaining critical path, longest first
NALAR_ROUTE_STATEFUL = 4     # problem flag: route a future to the instance of its type holding its state
NALAR_ROUTE_GREEDY = 8       # problem flag: route in output order with running instance loads
NALAR_ORDER_SRTF = 16        # problem flag: order by remaining critical path, shortest first
NALAR_ROUTE_WEIGHTED = 32    # problem flag: deal each type's futures to its instances by weight
NALAR_FORCE_GLOBAL_SWEEP = 1
NALAR_FORCE_TILED_SORT = 2
NALAR_FORCE_LEVEL_SWEEP = 4
NALAR_MAX_INSTANCES = 1024
NALAR_STATIC_MAX_NODES = 1 << 18       # largest snapshot of nalar_policy_pass_static
NALAR_STATIC_MAX_WORKFLOWS = 1 << 18

# why a graph-store pass was a full one (nalar_store_last_fallback)
NALAR_STORE_FULL_DISABLED = 1
NALAR_STORE_FULL_NO_STATE = 2
NALAR_STORE_FULL_SHRUNK = 3
NALAR_STORE_FULL_NO_SPLITTERS = 4
NALAR_STORE_FULL_OVERFLOW = 5
NALAR_STORE_FULL_ROUNDS = 6

EXPORTED = ("nalar_policy_create", "nalar_policy_pass", "nalar_policy_destroy", "nalar_policy_decide",
            "nalar_policy_pass_static",
            "nalar_policy_last_error", "nalar_policy_set_timing", "nalar_policy_get_timing",
            "nalar_store_create", "nalar_store_destroy", "nalar_store_append", "nalar_store_complete",
            "nalar_store_set_workflows", "nalar_store_set_instances", "nalar_store_n_nodes",
            "nalar_store_pass", "nalar_store_set_incremental", "nalar_store_last_pass_incremental",
            "nalar_store_last_fallback")


class NalarPolicyConfig(ctypes.Structure):
    _fields_ = [("device", ctypes.c_int32), ("flags", ctypes.c_uint32),
                ("stream", ctypes.c_void_p), ("reserve_nodes", ctypes.c_int64),
                ("reserve_edges", ctypes.c_int64), ("reserve_workflows", ctypes.c_int64)]


class NalarProblem(ctypes.Structure):
    _fields_ = [("n_nodes", ctypes.c_int64), ("n_edges", ctypes.c_int64),
                ("n_workflows", ctypes.c_int64), ("n_instances", ctypes.c_int64),
                ("now_us", ctypes.c_int64), ("migration_cost_us", ctypes.c_int64),
                ("flags", ctypes.c_uint32), ("reserved", ctypes.c_uint32),
                ("wf", ctypes.c_void_p), ("type", ctypes.c_void_p), ("est_us", ctypes.c_void_p),
                ("done", ctypes.c_void_p), ("loc", ctypes.c_void_p), ("dep_off", ctypes.c_void_p),
                ("dep_idx", ctypes.c_void_p), ("deadline_us", ctypes.c_void_p),
                ("inst_type", ctypes.c_void_p), ("inst_load_us", ctypes.c_void_p),
                ("inst_speed_permille", ctypes.c_void_p), ("wf_priority", ctypes.c_void_p),
                ("inst_weight", ctypes.c_void_p)]


class NalarResult(ctypes.Structure):
    _fields_ = [("rem_us", ctypes.c_void_p), ("order", ctypes.c_void_p),
                ("slack_us", ctypes.c_void_p), ("route", ctypes.c_void_p),
                ("cost_us", ctypes.c_void_p), ("n_ready", ctypes.c_int64)]


class NalarView(ctypes.Structure):
    _fields_ = [("rem_us", ctypes.c_void_p), ("order", ctypes.c_void_p),
                ("slack_us", ctypes.c_void_p), ("n_order", ctypes.c_int64)]


class NalarDecisions(ctypes.Structure):
    _fields_ = [("slack_us", ctypes.c_void_p), ("route", ctypes.c_void_p),
                ("cost_us", ctypes.c_void_p), ("rank", ctypes.c_void_p)]


_lib: Optional[ctypes.CDLL] = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with "
                           "`python -m paper_2601_05109_amd.build` (hipcc, gfx950)")
    lib = ctypes.CDLL(path)
    H = ctypes.c_void_p
    lib.nalar_policy_create.argtypes = [ctypes.POINTER(NalarPolicyConfig), ctypes.POINTER(H)]
    lib.nalar_policy_create.restype = ctypes.c_int
    lib.nalar_policy_pass.argtypes = [H, ctypes.POINTER(NalarProblem), ctypes.POINTER(NalarResult)]
    lib.nalar_policy_pass.restype = ctypes.c_int
    lib.nalar_policy_pass_static.argtypes = [H, ctypes.POINTER(NalarProblem), ctypes.POINTER(NalarResult)]
    lib.nalar_policy_pass_static.restype = ctypes.c_int
    lib.nalar_policy_decide.argtypes = [H, ctypes.POINTER(NalarProblem), ctypes.POINTER(NalarView),
                                        ctypes.c_int64, ctypes.c_void_p, ctypes.POINTER(NalarDecisions)]
    lib.nalar_policy_decide.restype = ctypes.c_int
    lib.nalar_policy_destroy.argtypes = [H]
    lib.nalar_policy_destroy.restype = None
    lib.nalar_policy_last_error.argtypes = [H]
    lib.nalar_policy_last_error.restype = ctypes.c_char_p
    lib.nalar_policy_set_timing.argtypes = [H, ctypes.c_int]
    lib.nalar_policy_set_timing.restype = ctypes.c_int
    lib.nalar_policy_get_timing.argtypes = [H, ctypes.POINTER(ctypes.c_char_p),
                                            ctypes.POINTER(ctypes.c_float), ctypes.c_int,
                                            ctypes.POINTER(ctypes.c_int)]
    lib.nalar_policy_get_timing.restype = ctypes.c_int
    P, I64, U32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint32
    lib.nalar_store_create.argtypes = [H, ctypes.POINTER(H)]
    lib.nalar_store_create.restype = ctypes.c_int
    lib.nalar_store_destroy.argtypes = [H]
    lib.nalar_store_destroy.restype = None
    lib.nalar_store_append.argtypes = [H, I64, I64, P, P, P, P, P, P, P, U32]
    lib.nalar_store_append.restype = ctypes.c_int
    lib.nalar_store_complete.argtypes = [H, I64, P]
    lib.nalar_store_complete.restype = ctypes.c_int
    lib.nalar_store_set_workflows.argtypes = [H, I64, P]
    lib.nalar_store_set_workflows.restype = ctypes.c_int
    lib.nalar_store_set_instances.argtypes = [H, I64, P, P, P]
    lib.nalar_store_set_instances.restype = ctypes.c_int
    lib.nalar_store_n_nodes.argtypes = [H]
    lib.nalar_store_n_nodes.restype = I64
    lib.nalar_store_pass.argtypes = [H, I64, I64, U32, ctypes.POINTER(NalarResult)]
    lib.nalar_store_pass.restype = ctypes.c_int
    lib.nalar_store_set_incremental.argtypes = [H, ctypes.c_int]
    lib.nalar_store_set_incremental.restype = ctypes.c_int
    lib.nalar_store_last_pass_incremental.argtypes = [H]
    lib.nalar_store_last_pass_incremental.restype = ctypes.c_int
    lib.nalar_store_last_fallback.argtypes = [H]
    lib.nalar_store_last_fallback.restype = ctypes.c_int
    _lib = lib
    return lib


# ---------------------------------------------------------------- C names

def nalar_policy_create(cfg: NalarPolicyConfig) -> tuple[int, Optional[int]]:
    h = ctypes.c_void_p()
    rc = load_library().nalar_policy_create(ctypes.byref(cfg), ctypes.byref(h))
    return rc, h.value


def nalar_policy_pass(h: int, prob: NalarProblem, res: NalarResult) -> int:
    return load_library().nalar_policy_pass(h, ctypes.byref(prob), ctypes.byref(res))


def nalar_policy_pass_static(h: int, prob: NalarProblem, res: NalarResult) -> int:
    return load_library().nalar_policy_pass_static(h, ctypes.byref(prob), ctypes.byref(res))


def nalar_policy_decide(h: int, prob: NalarProblem, view: NalarView, n_events: int, events,
                        out: NalarDecisions) -> int:
    return load_library().nalar_policy_decide(h, ctypes.byref(prob), ctypes.byref(view), n_events,
                                              events, ctypes.byref(out))


def nalar_policy_destroy(h: Optional[int]) -> None:
    load_library().nalar_policy_destroy(h)


def nalar_policy_last_error(h: Optional[int]) -> str:
    return (load_library().nalar_policy_last_error(h) or b"").decode()


def nalar_policy_set_timing(h: int, enable: bool) -> int:
    return load_library().nalar_policy_set_timing(h, 1 if enable else 0)


def nalar_policy_get_timing(h: int, cap: int = 32) -> list[tuple[str, float]]:
    names = (ctypes.c_char_p * cap)()
    ms = (ctypes.c_float * cap)()
    count = ctypes.c_int(0)
    rc = load_library().nalar_policy_get_timing(h, names, ms, cap, ctypes.byref(count))
    if rc != NALAR_OK:
        raise RuntimeError("no timed pass available")
    return [(names[i].decode(), float(ms[i])) for i in range(min(count.value, cap))]


def nalar_store_create(h: int) -> tuple[int, Optional[int]]:
    s = ctypes.c_void_p()
    rc = load_library().nalar_store_create(h, ctypes.byref(s))
    return rc, s.value


def nalar_store_destroy(s: Optional[int]) -> None:
    load_library().nalar_store_destroy(s)


def nalar_store_append(s: int, n_new: int, n_new_edges: int, wf, type, est_us, done, loc, dep_off,
                       dep_idx, flags: int = 0) -> int:
    return load_library().nalar_store_append(s, n_new, n_new_edges, wf, type, est_us, done, loc,
                                             dep_off, dep_idx, flags)


def nalar_store_complete(s: int, n: int, ids) -> int:
    return load_library().nalar_store_complete(s, n, ids)


def nalar_store_set_workflows(s: int, n_workflows: int, deadline_us) -> int:
    return load_library().nalar_store_set_workflows(s, n_workflows, deadline_us)


def nalar_store_set_instances(s: int, n_instances: int, inst_type, inst_load_us,
                              inst_speed_permille) -> int:
    return load_library().nalar_store_set_instances(s, n_instances, inst_type, inst_load_us,
                                                    inst_speed_permille)


def nalar_store_n_nodes(s: Optional[int]) -> int:
    return int(load_library().nalar_store_n_nodes(s))


def nalar_store_pass(s: int, now_us: int, migration_cost_us: int, policy: int, res: NalarResult) -> int:
    return load_library().nalar_store_pass(s, now_us, migration_cost_us, policy, ctypes.byref(res))


def nalar_store_set_incremental(s: Optional[int], enable: int) -> int:
    return load_library().nalar_store_set_incremental(s, enable)


def nalar_store_last_pass_incremental(s: Optional[int]) -> int:
    return int(load_library().nalar_store_last_pass_incremental(s))


def nalar_store_last_fallback(s: Optional[int]) -> int:
    return int(load_library().nalar_store_last_fallback(s))


# ---------------------------------------------------------------- torch helpers

class NalarError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"nalar_policy_pass returned {code}: {msg}")
        self.code = code


@dataclass
class DeviceProblem:
    """A snapshot held in device memory as torch tensors (plus the host scalars)."""
    now_us: int
    migration_cost_us: int
    wf_contiguous: bool
    tensors: dict

    FIELDS = ("wf", "type", "est_us", "done", "loc", "dep_off", "dep_idx", "deadline_us",
              "inst_type", "inst_load_us", "inst_speed_permille")

    @classmethod
    def from_host(cls, p, device="cuda") -> "DeviceProblem":
        import torch
        t = {}
        for f in cls.FIELDS:
            a = getattr(p, f)
            t[f] = torch.from_numpy(a.copy() if not a.flags.c_contiguous else a).to(device)
        return cls(int(p.now_us), int(p.migration_cost_us), bool(p.wf_contiguous), t)

    @property
    def n_nodes(self) -> int:
        return int(self.tensors["wf"].shape[0])

    def c_struct(self, flags: Optional[int] = None, policy: int = 0, priority=None,
                 weights=None) -> NalarProblem:
        """The C struct of this problem.  ``flags`` replaces the default
        problem flags (the contiguity bit when the ids are workflow-contiguous);
        ``policy`` (NALAR_ORDER_* and NALAR_ROUTE_* bits) is ORed in;
        ``priority`` is a uint8 device tensor of one level per workflow, or
        None; ``weights`` a uint32 (or int32) device tensor of one routing
        weight per instance, or None."""
        t = self.tensors
        ptr = lambda x: x.data_ptr() if x.numel() > 0 else None
        return NalarProblem(
            n_nodes=t["wf"].shape[0], n_edges=t["dep_idx"].shape[0],
            n_workflows=t["deadline_us"].shape[0], n_instances=t["inst_type"].shape[0],
            now_us=self.now_us, migration_cost_us=self.migration_cost_us,
            flags=((NALAR_WF_CONTIGUOUS if self.wf_contiguous else 0) if flags is None else flags) | policy,
            reserved=0, wf=ptr(t["wf"]), type=ptr(t["type"]), est_us=ptr(t["est_us"]),
            done=ptr(t["done"]), loc=ptr(t["loc"]), dep_off=ptr(t["dep_off"]),
            dep_idx=ptr(t["dep_idx"]), deadline_us=ptr(t["deadline_us"]),
            inst_type=ptr(t["inst_type"]), inst_load_us=ptr(t["inst_load_us"]),
            inst_speed_permille=ptr(t["inst_speed_permille"]),
            wf_priority=None if priority is None else priority.data_ptr(),
            inst_weight=None if weights is None else weights.data_ptr())


@dataclass
class DeviceResult:
    rem: object
    order: object
    slack: object
    route: object
    cost: object
    n_ready: int = 0

    @classmethod
    def alloc(cls, n: int, device="cuda", rem: bool = True, cost: bool = True) -> "DeviceResult":
        import torch
        n1 = max(n, 1)
        return cls(torch.empty(n1, dtype=torch.int64, device=device) if rem else None,
                   torch.empty(n1, dtype=torch.int32, device=device),
                   torch.empty(n1, dtype=torch.int64, device=device),
                   torch.empty(n1, dtype=torch.int32, device=device),
                   torch.empty(n1, dtype=torch.int64, device=device) if cost else None)

    def c_struct(self) -> NalarResult:
        p = lambda x: None if x is None else x.data_ptr()
        return NalarResult(rem_us=p(self.rem), order=p(self.order), slack_us=p(self.slack),
                           route=p(self.route), cost_us=p(self.cost), n_ready=0)


# Handles still open when the interpreter exits are closed by an atexit hook,
# which runs before modules are torn down: the library's device and pinned
# memory is then released while the HIP runtime (and a profiler attached to
# it) is fully alive, and no library call is left for interpreter
# finalization or the C exit handlers.  Objects collected during
# finalization do not call the library at all.
_open_handles: "weakref.WeakSet" = weakref.WeakSet()


@atexit.register
def _close_open_handles() -> None:
    for obj in sorted(list(_open_handles), key=lambda o: 0 if isinstance(o, Store) else 1):
        try:
            obj.close()
        except Exception:
            pass


@dataclass
class DeviceDecisions:
    """Outputs of per-event decisions: one entry per event."""
    slack: object
    route: object
    cost: object
    rank: object

    @classmethod
    def alloc(cls, n: int, device="cuda") -> "DeviceDecisions":
        import torch
        n1 = max(n, 1)
        return cls(torch.empty(n1, dtype=torch.int64, device=device),
                   torch.empty(n1, dtype=torch.int32, device=device),
                   torch.empty(n1, dtype=torch.int64, device=device),
                   torch.empty(n1, dtype=torch.int64, device=device))

    def c_struct(self) -> NalarDecisions:
        p = lambda x: None if x is None else x.data_ptr()
        return NalarDecisions(slack_us=p(self.slack), route=p(self.route), cost_us=p(self.cost),
                              rank=p(self.rank))


class Policy:
    """Owns one handle bound to a device and a stream."""

    def __init__(self, device: int = 0, stream=None, flags: int = 0, reserve_nodes: int = 0,
                 reserve_workflows: int = 0):
        import torch
        if stream is None:
            stream = torch.cuda.current_stream(device)
        self.stream = stream
        cfg = NalarPolicyConfig(device=device, flags=flags, stream=stream.cuda_stream,
                                reserve_nodes=reserve_nodes, reserve_edges=0,
                                reserve_workflows=reserve_workflows)
        rc, h = nalar_policy_create(cfg)
        if rc != NALAR_OK:
            raise NalarError(rc, nalar_policy_last_error(None))
        self.handle = h
        _open_handles.add(self)

    def close(self) -> None:
        if self.handle:
            nalar_policy_destroy(self.handle)
            self.handle = None
        _open_handles.discard(self)

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        # closed already, or the interpreter (and maybe the runtime) going away:
        # leave it to process exit (module globals such as sys may be gone)
        if getattr(self, "handle", None) is None or _is_finalizing():
            return
        try:
            self.close()
        except Exception:
            pass

    def run_pass(self, prob: DeviceProblem, out: DeviceResult, flags: Optional[int] = None,
                 raw: Optional[NalarProblem] = None, policy: int = 0, priority=None) -> int:
        """One synchronous pass; returns the C return code and fills out.n_ready."""
        cp = raw if raw is not None else prob.c_struct(flags, policy, priority)
        cr = out.c_struct()
        rc = nalar_policy_pass(self.handle, cp, cr)
        out.n_ready = int(cr.n_ready) if rc == NALAR_OK else 0
        return rc

    def decide(self, prob: DeviceProblem, view: "DeviceResult", events, out: "DeviceDecisions",
               flags: Optional[int] = None, policy: int = 0, priority=None,
               raw: Optional[NalarProblem] = None) -> int:
        """Decide the futures of ``events`` (an int32 device tensor) against the
        view a pass left in ``view`` (its rem, order and slack, n_ready
        entries); fills ``out`` (one entry per event).  Synchronous."""
        cp = raw if raw is not None else prob.c_struct(flags, policy, priority)
        cv = NalarView(rem_us=view.rem.data_ptr(), order=view.order.data_ptr(),
                       slack_us=view.slack.data_ptr(), n_order=view.n_ready)
        n = int(events.shape[0])
        return nalar_policy_decide(self.handle, cp, cv, n, events.data_ptr() if n else None,
                                   out.c_struct())

    def last_error(self) -> str:
        return nalar_policy_last_error(self.handle)

    def set_timing(self, enable: bool) -> None:
        nalar_policy_set_timing(self.handle, enable)

    def timing(self) -> list[tuple[str, float]]:
        return nalar_policy_get_timing(self.handle)


class Store:
    """A device-resident graph store bound to a Policy: the snapshot is kept in
    HBM across passes and updated by deltas (arrays are torch device tensors
    or numpy arrays, uploaded first).  Copies are enqueued on the policy's
    stream, which is the stream torch allocated the tensors on, so a tensor may
    be dropped right after the call."""

    def __init__(self, policy: "Policy"):
        rc, h = nalar_store_create(policy.handle)
        if rc != NALAR_OK:
            raise NalarError(rc, policy.last_error())
        self.policy = policy
        self.handle = h
        _open_handles.add(self)

    @staticmethod
    def _dev(a, dtype, device="cuda"):
        import numpy as np
        import torch
        if isinstance(a, np.ndarray):
            a = torch.from_numpy(np.ascontiguousarray(a.astype(dtype, copy=False))).to(device)
        return a

    @staticmethod
    def _ptr(t):
        return t.data_ptr() if t is not None and t.numel() > 0 else None

    def append(self, wf, type, est_us, done, loc, dep_off, dep_idx, contiguous: bool = False) -> int:
        import numpy as np
        t = [self._dev(a, d) for a, d in ((wf, np.int32), (type, np.int32), (est_us, np.int64),
                                          (done, np.uint8), (loc, np.int32), (dep_off, np.int32),
                                          (dep_idx, np.int32))]
        n, e = int(t[0].shape[0]), int(t[6].shape[0])
        return nalar_store_append(self.handle, n, e, *[self._ptr(x) for x in t],
                                  NALAR_WF_CONTIGUOUS if contiguous else 0)

    def complete(self, ids) -> int:
        import numpy as np
        t = self._dev(ids, np.int32)
        return nalar_store_complete(self.handle, int(t.shape[0]), self._ptr(t))

    def set_workflows(self, deadline_us) -> int:
        import numpy as np
        t = self._dev(deadline_us, np.int64)
        return nalar_store_set_workflows(self.handle, int(t.shape[0]), self._ptr(t))

    def set_instances(self, inst_type, inst_load_us, inst_speed_permille) -> int:
        import numpy as np
        t = [self._dev(inst_type, np.int32), self._dev(inst_load_us, np.int64),
             self._dev(inst_speed_permille, np.int32)]
        return nalar_store_set_instances(self.handle, int(t[0].shape[0]), *[self._ptr(x) for x in t])

    @property
    def n_nodes(self) -> int:
        return nalar_store_n_nodes(self.handle)

    def set_incremental(self, enable: bool) -> int:
        return nalar_store_set_incremental(self.handle, 1 if enable else 0)

    @property
    def last_pass_incremental(self) -> bool:
        return nalar_store_last_pass_incremental(self.handle) == 1

    @property
    def last_fallback(self) -> int:
        """0 after an incremental pass, else a NALAR_STORE_FULL_* reason."""
        return nalar_store_last_fallback(self.handle)

    def run_pass(self, out: "DeviceResult", now_us: int, migration_cost_us: int, policy: int = 0) -> int:
        cr = out.c_struct()
        rc = nalar_store_pass(self.handle, now_us, migration_cost_us, policy, cr)
        out.n_ready = int(cr.n_ready) if rc == NALAR_OK else 0
        return rc

    def close(self) -> None:
        if self.handle:
            nalar_store_destroy(self.handle)
            self.handle = None
        _open_handles.discard(self)

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        if getattr(self, "handle", None) is None or _is_finalizing():
            return
        try:
            self.close()
        except Exception:
            pass


def run(p, device: str = "cuda", policy: Optional[Policy] = None, flags: int = 0):
    """Upload a host problem, run one pass, and return host numpy results:
    (status, n_ready, rem, order, slack, route, cost)."""
    dp = DeviceProblem.from_host(p, device)
    out = DeviceResult.alloc(dp.n_nodes, device)
    own = policy is None
    pol = policy or Policy(flags=flags)
    try:
        rc = pol.run_pass(dp, out)
    finally:
        if own:
            pol.close()
    R = out.n_ready
    N = dp.n_nodes
    return (rc, R, out.rem[:N].cpu().numpy(), out.order[:R].cpu().numpy(),
            out.slack[:R].cpu().numpy(), out.route[:R].cpu().numpy(), out.cost[:R].cpu().numpy())
