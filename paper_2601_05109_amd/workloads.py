"""Seeded synthetic inputs for the global policy pass.

This module only *generates* problems: dependency graphs of in-flight futures,
their attributes, workflow deadlines and the component-instance table.  It
holds none of the pass's arithmetic (no remaining-path, slack, ordering or
routing computation), so that the CPU oracle and the HIP path can both consume
its arrays without sharing any code of the method.

The shapes and value distributions stand in for the paper's emulated
scalability workload (Section 6.3: 1,024 to 131K futures, profiled LLM call
latencies replacing inference, 64/128 agents).  Every array is int64 for time
values (fixed-point microseconds), int32 for ids and offsets, uint8 for flags.

Generators
----------
``tiny(seed)``          64 workflows x 32 futures, K=4 types, 16 instances.
``paper_scale(seed)``   4,096 x 32 = 131,072 futures, K=8, 64 instances.
``deep_chains(seed)``   1,024 x 512 futures, 128 layers of width 4, K=8, 128 inst.
``wide_mapreduce(seed)`` 256 x (1 root + 4,096 tools + 1 reduce), K=8, 256 inst.
``dynamic_stream(...)``  the wide map/reduce graph evolved over 100 steps.
``churned(p, seed)``    p with 1 % of its in-flight futures completed.
``deadline_shifted(p, seed)`` p with every deadline moved by up to 1 s.
``random_dag(seed,...)`` small arbitrary DAGs for brute-force checks.
``relabel(p, perm)``    the same problem under a permutation of node ids.
"""
from __future__ import annotations

import dataclasses
import hashlib
from typing import Iterator, Optional

import numpy as np

NOW_US = 1_767_225_600_000_000          # fixed "now" of every synthetic snapshot
MIGRATION_COST_US = 200_000             # state-migration penalty of every workload
EST_MAX_US = 1 << 40                    # largest service-time estimate accepted
SEED_BASE = 260105109

LLM_MU, LLM_SIGMA = float(np.log(800_000.0)), 0.6     # LLM component types (k < 2)
TOOL_MU, TOOL_SIGMA = float(np.log(50_000.0)), 1.0     # tool component types


@dataclasses.dataclass
class Problem:
    """One snapshot of the global view: futures, workflows and instances.

    Node arrays have length ``n_nodes``; ``dep_off``/``dep_idx`` is the
    dependency (parent) CSR; ``deadline_us`` has one entry per workflow and the
    ``inst_*`` arrays one entry per component instance.  ``wf_contiguous`` is
    True when the nodes of each workflow occupy one contiguous, ascending id
    range in workflow order (the layout hint of the C ABI).
    """
    name: str
    now_us: int
    migration_cost_us: int
    wf: np.ndarray
    type: np.ndarray
    est_us: np.ndarray
    done: np.ndarray
    loc: np.ndarray
    dep_off: np.ndarray
    dep_idx: np.ndarray
    deadline_us: np.ndarray
    inst_type: np.ndarray
    inst_load_us: np.ndarray
    inst_speed_permille: np.ndarray
    wf_contiguous: bool = False

    @property
    def n_nodes(self) -> int:
        return int(self.wf.shape[0])

    @property
    def n_edges(self) -> int:
        return int(self.dep_idx.shape[0])

    @property
    def n_workflows(self) -> int:
        return int(self.deadline_us.shape[0])

    @property
    def n_instances(self) -> int:
        return int(self.inst_type.shape[0])

    NODE_FIELDS = ("wf", "type", "est_us", "done", "loc")
    ARRAY_FIELDS = ("wf", "type", "est_us", "done", "loc", "dep_off", "dep_idx",
                    "deadline_us", "inst_type", "inst_load_us", "inst_speed_permille")
    DTYPES = {"wf": np.int32, "type": np.int32, "est_us": np.int64, "done": np.uint8,
              "loc": np.int32, "dep_off": np.int32, "dep_idx": np.int32,
              "deadline_us": np.int64, "inst_type": np.int32, "inst_load_us": np.int64,
              "inst_speed_permille": np.int32}

    def check_dtypes(self) -> None:
        for f in self.ARRAY_FIELDS:
            a = getattr(self, f)
            if a.dtype != self.DTYPES[f] or not a.flags.c_contiguous:
                raise TypeError(f"{f}: expected contiguous {self.DTYPES[f]}, got {a.dtype}")

    def copy(self, **changes) -> "Problem":
        kw = {f.name: getattr(self, f.name) for f in dataclasses.fields(self)}
        for f in self.ARRAY_FIELDS:
            kw[f] = np.array(kw[f], copy=True)
        kw.update(changes)
        return Problem(**kw)

    def digest(self) -> dict:
        """SHA-256 (first 16 hex digits) of every array, for reports."""
        out = {}
        for f in self.ARRAY_FIELDS:
            out[f] = hashlib.sha256(np.ascontiguousarray(getattr(self, f)).tobytes()).hexdigest()[:16]
        return out


# ---------------------------------------------------------------------------
# shared samplers (input distributions only)
# ---------------------------------------------------------------------------

def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def _est_for_types(rng: np.random.Generator, types: np.ndarray) -> np.ndarray:
    """Service-time estimates: lognormal per component class, rounded half-up,
    clamped to [1, 2^40] microseconds."""
    llm = types < 2
    mu = np.where(llm, LLM_MU, TOOL_MU)
    sigma = np.where(llm, LLM_SIGMA, TOOL_SIGMA)
    x = rng.lognormal(mean=mu, sigma=sigma)
    return np.clip(np.floor(x + 0.5), 1, EST_MAX_US).astype(np.int64)


def _loc(rng: np.random.Generator, n: int, m: int) -> np.ndarray:
    """Managed-state location: an instance id with probability 1/2, else -1."""
    has = rng.random(n) < 0.5
    ids = rng.integers(0, m, size=n) if m > 0 else np.zeros(n, np.int64)
    return np.where(has, ids, -1).astype(np.int32)


def _instances(rng: np.random.Generator, m: int, k: int):
    inst_type = rng.integers(0, k, size=m).astype(np.int32)
    load = rng.integers(0, 2_000_000, size=m, endpoint=True).astype(np.int64)
    speed = rng.integers(500, 2000, size=m, endpoint=True).astype(np.int32)
    return inst_type, load, speed


def _deadlines(rng: np.random.Generator, w: int, now: int) -> np.ndarray:
    return (now + rng.integers(2_000_000, 20_000_000, size=w, endpoint=True)).astype(np.int64)


def _csr_from_counts(counts: np.ndarray, parents: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    off = np.zeros(counts.shape[0] + 1, np.int64)
    np.cumsum(counts, out=off[1:])
    if off[-1] >= 2**31:
        raise ValueError("edge count exceeds int32 offsets")
    return off.astype(np.int32), parents.astype(np.int32)


def _pick_distinct(rng: np.random.Generator, window: np.ndarray, count: np.ndarray,
                   width: int) -> tuple[np.ndarray, np.ndarray]:
    """For each row r choose count[r] distinct columns of range(window[r]) uniformly.

    Returns (row_index, column) pairs in ascending (row, column) order."""
    keys = rng.random((window.shape[0], width))
    keys[np.arange(width)[None, :] >= window[:, None]] = np.inf
    order = np.argsort(keys, axis=1, kind="stable")
    take = np.arange(width)[None, :] < count[:, None]
    rows = np.nonzero(take)[0]
    cols = order[take]
    # sort columns within each row ascending (canonical dependency order)
    srt = np.lexsort((cols, rows))
    return rows[srt], cols[srt]


def _windowed(name: str, seed: int, W: int, n: int, K: int, M: int) -> Problem:
    """Workflows of n topologically indexed futures; node i>0 draws
    1+min(Poisson(0.5),2) distinct parents from the previous 8 nodes; the first
    30% of each workflow is done."""
    rng = _rng(seed)
    N = W * n
    local = np.tile(np.arange(n, dtype=np.int64), W)
    wf = np.repeat(np.arange(W, dtype=np.int64), n)
    pois = rng.poisson(0.5, size=N)
    window = np.minimum(local, 8)
    count = np.minimum(1 + np.minimum(pois, 2), window)
    rows, cols = _pick_distinct(rng, window, count, 8)
    parent_local = local[rows] - window[rows] + cols
    parents = wf[rows] * n + parent_local
    dep_off, dep_idx = _csr_from_counts(count, parents)
    types = rng.integers(0, K, size=N).astype(np.int32)
    est = _est_for_types(rng, types)
    done = (local < (3 * n) // 10).astype(np.uint8)
    loc = _loc(rng, N, M)
    deadline = _deadlines(rng, W, NOW_US)
    it, il, isp = _instances(rng, M, K)
    return Problem(name, NOW_US, MIGRATION_COST_US, wf.astype(np.int32), types, est, done,
                   loc, dep_off, dep_idx, deadline, it, il, isp, wf_contiguous=True)


def tiny(seed: Optional[int] = None) -> Problem:
    """64 workflows x 32 futures (2,048 nodes), K=4, 16 instances."""
    return _windowed("tiny-64x32", SEED_BASE + 0 if seed is None else seed, 64, 32, 4, 16)


def paper_scale(seed: Optional[int] = None) -> Problem:
    """4,096 workflows x 32 futures = 131,072 futures, K=8, 64 instances."""
    return _windowed("paper-scale-4096x32", SEED_BASE + 1 if seed is None else seed,
                     4096, 32, 8, 64)


def windowed(W: int, seed: Optional[int] = None) -> Problem:
    """W workflows x 32 futures from the paper-scale generator (K=8, 64
    instances): the futures-count sweep of the scalability study."""
    return _windowed(f"windowed-{W}x32", SEED_BASE + 1 if seed is None else seed, W, 32, 8, 64)


def deep_chains(seed: Optional[int] = None, W: int = 1024) -> Problem:
    """1,024 workflows x 512 futures: 128 layers of width 4, each node with 1-3
    distinct parents in the previous layer; K=8, 128 instances."""
    rng = _rng(SEED_BASE + 2 if seed is None else seed)
    n, width, K, M = 512, 4, 8, 128
    N = W * n
    local = np.tile(np.arange(n, dtype=np.int64), W)
    wf = np.repeat(np.arange(W, dtype=np.int64), n)
    layer = local // width
    count = np.where(layer > 0, rng.integers(1, 4, size=N), 0)
    window = np.where(layer > 0, width, 0)
    rows, cols = _pick_distinct(rng, window, count, width)
    parents = wf[rows] * n + (layer[rows] - 1) * width + cols
    dep_off, dep_idx = _csr_from_counts(count, parents)
    types = rng.integers(0, K, size=N).astype(np.int32)
    est = _est_for_types(rng, types)
    done = (local < (3 * n) // 10).astype(np.uint8)
    loc = _loc(rng, N, M)
    deadline = _deadlines(rng, W, NOW_US)
    it, il, isp = _instances(rng, M, K)
    return Problem(f"deep-chains-{W}x512", NOW_US, MIGRATION_COST_US, wf.astype(np.int32),
                   types, est, done, loc, dep_off, dep_idx, deadline, it, il, isp,
                   wf_contiguous=True)


def wide_mapreduce(seed: Optional[int] = None, W: int = 256, fan: int = 4096) -> Problem:
    """W workflows, each 1 root LLM (done) -> ``fan`` tool futures -> 1 reduce LLM;
    K=8, 256 instances."""
    rng = _rng(SEED_BASE + 3 if seed is None else seed)
    n, K, M = fan + 2, 8, 256
    N = W * n
    local = np.tile(np.arange(n, dtype=np.int64), W)
    wf = np.repeat(np.arange(W, dtype=np.int64), n)
    base = np.arange(W, dtype=np.int64) * n
    is_tool = (local >= 1) & (local <= fan)
    is_red = local == fan + 1
    count = np.where(is_tool, 1, np.where(is_red, fan, 0)).astype(np.int64)
    # dependency lists in node order: tools -> {root}; reduce -> {tools}
    per_wf = np.concatenate([np.zeros(fan, np.int64), np.arange(1, fan + 1, dtype=np.int64)])
    parents = (base[:, None] + per_wf[None, :]).reshape(-1)
    dep_off, dep_idx = _csr_from_counts(count, parents)
    types = np.where(is_tool, rng.integers(2, K, size=N), rng.integers(0, 2, size=N)).astype(np.int32)
    est = _est_for_types(rng, types)
    done = (local == 0).astype(np.uint8)
    loc = _loc(rng, N, M)
    deadline = _deadlines(rng, W, NOW_US)
    it, il, isp = _instances(rng, M, K)
    return Problem(f"wide-mapreduce-{W}x{n}", NOW_US, MIGRATION_COST_US, wf.astype(np.int32),
                   types, est, done, loc, dep_off, dep_idx, deadline, it, il, isp,
                   wf_contiguous=True)


# ---------------------------------------------------------------------------
# dynamic stream: the wide map/reduce graph evolving over steps
# ---------------------------------------------------------------------------

class _Growable:
    def __init__(self, a: np.ndarray, cap: int):
        self.buf = np.empty(max(cap, a.shape[0]), a.dtype)
        self.buf[: a.shape[0]] = a
        self.n = a.shape[0]

    def extend(self, b: np.ndarray) -> None:
        need = self.n + b.shape[0]
        if need > self.buf.shape[0]:
            nb = np.empty(max(need, int(self.buf.shape[0] * 1.5)), self.buf.dtype)
            nb[: self.n] = self.buf[: self.n]
            self.buf = nb
        self.buf[self.n: need] = b
        self.n = need

    @property
    def view(self) -> np.ndarray:
        return self.buf[: self.n]


def dynamic_stream(steps: int = 100, seed: Optional[int] = None, W: int = 256,
                   fan: int = 4096, growth: str = "compound") -> Iterator[Problem]:
    """Yield snapshots 0..steps of an evolving wide map/reduce graph.

    Snapshot 0 is ``wide_mapreduce(W=W, fan=fan)``.  Each later step, with its own
    generator seeded from ``SeedSequence([seed, step])``:

    1. ``floor(R/100)`` running futures complete, uniformly without replacement,
       where "running" means dispatched and not yet done, i.e. not done and all
       of its parents done (the simulation tracks this with its own
       pending-parent counters, as a component controller would);
    2. ``floor(N/100)`` distinct nodes, uniform over all current nodes (with
       ``growth="compound"``; ``"linear"`` uses the original N instead), each
       append 1-4 new child futures with that node as their only dependency, the
       same workflow, a uniform type in [0, K), service times and state location
       from the tiny/paper-scale distributions, not done; new ids are appended in
       ascending (parent, j) order, so workflows stop being contiguous.

    The yielded arrays are views into growing buffers: a snapshot is valid until
    the iterator advances (copy it to keep it).  Evolution never reads a pass
    output; ``now`` and the instance table stay fixed.
    """
    seed4 = SEED_BASE + 4 if seed is None else seed
    p0 = wide_mapreduce(W=W, fan=fan)
    n0 = p0.n_nodes
    K, M = 8, p0.n_instances
    cap = int(n0 * 13) if growth == "compound" else int(n0 * 4)
    wf = _Growable(p0.wf, cap)
    ty = _Growable(p0.type, cap)
    est = _Growable(p0.est_us, cap)
    done = _Growable(p0.done, cap)
    loc = _Growable(p0.loc, cap)
    dep_off = _Growable(p0.dep_off, cap + 1)
    dep_idx = _Growable(p0.dep_idx, cap + n0)
    # simulation bookkeeping: pending (not-done) parent counts and children of
    # appended nodes (each appended node has exactly one parent)
    pending = _Growable(np.zeros(n0, np.int64), cap)
    n = fan + 2
    local0 = np.tile(np.arange(n), W)
    pending.buf[:n0] = np.where((local0 >= 1) & (local0 <= fan), 0,
                                np.where(local0 == fan + 1, fan, 0))
    reduce_of_wf = np.arange(W, dtype=np.int64) * n + fan + 1
    app_parent = _Growable(np.zeros(0, np.int64), cap)   # parent of node n0 + j
    running = _Growable(((done.view == 0) & (pending.view == 0)).astype(np.bool_), cap)

    def snapshot(step: int) -> Problem:
        N = wf.n
        return Problem(f"dynamic-step{step}", NOW_US, MIGRATION_COST_US, wf.view, ty.view,
                       est.view, done.view, loc.view, dep_off.view, dep_idx.view,
                       p0.deadline_us, p0.inst_type, p0.inst_load_us, p0.inst_speed_permille,
                       wf_contiguous=(N == n0))

    yield snapshot(0)
    for step in range(1, steps + 1):
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed4, step])))
        N = wf.n
        # (1) completions among running futures
        run_ids = np.flatnonzero(running.view)
        k = run_ids.shape[0] // 100
        if k > 0:
            fin = np.sort(rng.choice(run_ids, size=k, replace=False))
            done.buf[fin] = 1
            running.buf[fin] = False
            # children of finished nodes: the per-workflow reduce (of tools) and
            # appended nodes whose only parent finished
            is_tool = (fin < n0) & (fin % n >= 1) & (fin % n <= fan)
            red = reduce_of_wf[fin[is_tool] // n]
            if red.shape[0]:
                np.subtract.at(pending.buf, red, 1)
                ready_red = red[(pending.buf[red] == 0) & (done.buf[red] == 0)]
                running.buf[ready_red] = True
            if app_parent.n:
                fin_mask = np.zeros(N, np.bool_)
                fin_mask[fin] = True
                kids = np.flatnonzero(fin_mask[app_parent.view]) + n0
                pending.buf[kids] -= 1
                ok = kids[(pending.buf[kids] == 0) & (done.buf[kids] == 0)]
                running.buf[ok] = True
        # (2) appends
        base_n = N if growth == "compound" else n0
        m = base_n // 100
        if m > 0:
            us = np.sort(rng.choice(N, size=m, replace=False))
            per = rng.integers(1, 5, size=m)
            par = np.repeat(us, per)
            t = par.shape[0]
            new_type = rng.integers(0, K, size=t).astype(np.int32)
            new_est = _est_for_types(rng, new_type)
            new_loc = _loc(rng, t, M)
            wf.extend(wf.view[par])
            ty.extend(new_type)
            est.extend(new_est)
            done.extend(np.zeros(t, np.uint8))
            loc.extend(new_loc)
            last = int(dep_off.view[-1])
            dep_off.extend((last + np.arange(1, t + 1)).astype(np.int32))
            dep_idx.extend(par.astype(np.int32))
            pend = (done.buf[par] == 0).astype(np.int64)
            pending.extend(pend)
            app_parent.extend(par)
            running.extend(pend == 0)
        yield snapshot(step)


def churned(p: Problem, seed: int, frac: float = 0.01) -> Problem:
    """p with ``frac`` of its not-done futures (uniform, without replacement)
    marked done: the values of 1 % of the in-flight futures materialised
    since the last snapshot."""
    rng = _rng(seed)
    live = np.flatnonzero(p.done == 0)
    k = int(live.shape[0] * frac)
    done = p.done.copy()
    if k > 0:
        done[rng.choice(live, size=k, replace=False)] = 1
    return p.copy(done=done)


def deadline_shifted(p: Problem, seed: int, max_shift_us: int = 1_000_000) -> Problem:
    """p with every workflow deadline moved by its own uniform shift in
    [-max_shift_us, max_shift_us] (deadlines renegotiated, clocks adjusted)."""
    rng = _rng(seed)
    shift = rng.integers(-max_shift_us, max_shift_us, size=p.n_workflows, endpoint=True)
    return p.copy(deadline_us=(p.deadline_us + shift).astype(np.int64))


# ---------------------------------------------------------------------------
# small arbitrary problems
# ---------------------------------------------------------------------------

def random_dag(seed: int, n_nodes: int = 8, n_workflows: int = 2, n_instances: int = 4,
               n_types: int = 3, p_edge: float = 0.35, p_done: float = 0.3,
               est_max: int = 50, load_max: int = 100, speed_lo: int = 1,
               speed_hi: int = 3000, mig: Optional[int] = None, dup_edges: bool = True,
               zero_est: float = 0.15, shuffle_ids: bool = True) -> Problem:
    """A small arbitrary DAG over several workflows, for exhaustive checks.

    Edges run only inside a workflow and from an earlier to a later node of a
    hidden topological order; ids are then shuffled (``shuffle_ids``) so neither
    topological nor workflow-contiguous indexing holds.  Duplicate dependencies,
    zero service times, done sets that are not ancestor-closed, instances of
    types no future has and futures of types no instance has all occur."""
    rng = _rng(seed)
    N, W, M = n_nodes, max(1, n_workflows), n_instances
    wf = np.sort(rng.integers(0, W, size=N))
    parents: list[list[int]] = [[] for _ in range(N)]
    for v in range(N):
        for u in range(v):
            if wf[u] == wf[v] and rng.random() < p_edge:
                parents[v].append(u)
                if dup_edges and rng.random() < 0.1:
                    parents[v].append(u)
    perm = rng.permutation(N) if shuffle_ids else np.arange(N)
    # perm[old] = new id
    new_par: list[list[int]] = [[] for _ in range(N)]
    for v in range(N):
        new_par[perm[v]] = [int(perm[u]) for u in parents[v]]
    wf_new = np.empty(N, np.int64)
    wf_new[perm] = wf
    counts = np.array([len(x) for x in new_par], np.int64)
    flat = np.array([u for x in new_par for u in x], np.int64)
    dep_off, dep_idx = _csr_from_counts(counts, flat)
    types = rng.integers(0, n_types + 1, size=N).astype(np.int32)
    est = rng.integers(0, est_max + 1, size=N).astype(np.int64)
    est[rng.random(N) < zero_est] = 0
    done = (rng.random(N) < p_done).astype(np.uint8)
    loc = np.where(rng.random(N) < 0.5, rng.integers(0, max(M, 1), size=N), -1).astype(np.int32)
    if M == 0:
        loc[:] = -1
    now = int(rng.integers(0, 1000))
    deadline = (now + rng.integers(-200, 400, size=W)).astype(np.int64)
    inst_type = rng.integers(0, n_types, size=M).astype(np.int32)
    load = rng.integers(0, load_max + 1, size=M).astype(np.int64)
    speed = rng.integers(speed_lo, speed_hi + 1, size=M).astype(np.int32)
    mig_us = int(rng.integers(0, 300)) if mig is None else mig
    return Problem(f"random-dag-{seed}", now, mig_us, wf_new.astype(np.int32), types, est, done,
                   loc, dep_off, dep_idx, deadline, inst_type, load, speed,
                   wf_contiguous=bool(np.all(np.diff(wf_new) >= 0)))


def relabel(p: Problem, perm: np.ndarray) -> Problem:
    """The same problem with node id v renamed perm[v] (perm a permutation).

    Dependency lists keep their per-node order.  The result is generally neither
    topologically indexed nor workflow-contiguous."""
    N = p.n_nodes
    perm = np.asarray(perm, np.int64)
    inv = np.empty(N, np.int64)
    inv[perm] = np.arange(N)
    out = {}
    for f in Problem.NODE_FIELDS:
        a = getattr(p, f)
        out[f] = np.ascontiguousarray(a[inv])
    counts = np.diff(p.dep_off.astype(np.int64))
    new_counts = counts[inv]
    starts = p.dep_off[:-1].astype(np.int64)[inv]
    new_off = np.zeros(N + 1, np.int64)
    np.cumsum(new_counts, out=new_off[1:])
    E = int(new_off[-1])
    idx = np.arange(E, dtype=np.int64) - np.repeat(new_off[:-1] - starts, new_counts)
    flat = perm[p.dep_idx.astype(np.int64)[idx]] if E else np.zeros(0, np.int64)
    dep_off, dep_idx = _csr_from_counts(new_counts, flat)
    contiguous = bool(np.all(np.diff(out["wf"].astype(np.int64)) >= 0))
    return Problem(p.name + "-relabelled", p.now_us, p.migration_cost_us, out["wf"], out["type"],
                   out["est_us"], out["done"], out["loc"], dep_off, dep_idx, p.deadline_us.copy(),
                   p.inst_type.copy(), p.inst_load_us.copy(), p.inst_speed_permille.copy(),
                   wf_contiguous=contiguous)


WORKLOADS = {
    "tiny": tiny,
    "paper-scale": paper_scale,
    "deep-chains": deep_chains,
    "wide-mapreduce": wide_mapreduce,
}
