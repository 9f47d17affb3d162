"""GPU parity of incremental passes over the graph store.

After a successful pass the store keeps every future's remaining critical
path; the next pass recomputes it only for the futures appended or completed
since and their ancestors (Section 4.3.1's dynamic graph), then keys, routes
and orders the ready futures afresh.  Every pass is checked bit-exactly
against the oracle on the full snapshot the deltas add up to, and the tests
assert that the incremental path actually ran:

- every step 0..100 of the evolving map/reduce stream, fed as deltas;
- growing random DAGs: several workflows appended interleaved (ids not
  grouped by workflow), futures with several dependencies, dependencies on
  futures appended later in the same call, futures with more dependencies
  than one thread expands, completions of any future, deadline and instance
  changes, every order and routing policy;
- incremental and full passes agree pass by pass on one delta stream;
- error rules: a cycle or a dependency on another workflow among appended
  futures, a dependency out of range, malformed appended offsets.
"""
import concurrent.futures as cf
import sys

import numpy as np
import pytest

import oracle
from paper_2601_05109_amd import workloads as wl
from test_gpu_parity import assert_parity, say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover - collected on CPU hosts too
    pytest.skip("no GPU", allow_module_level=True)

from paper_2601_05109_amd import nalar  # noqa: E402


def store_pass(pol, st, p, policy=0):
    out = nalar.DeviceResult.alloc(max(p.n_nodes, 1))
    rc = st.run_pass(out, p.now_us, p.migration_cost_us, policy=policy)
    torch.cuda.synchronize()
    R = out.n_ready
    return dict(status=rc, n_ready=R, rem=out.rem[:p.n_nodes].cpu().numpy(),
                order=out.order[:R].cpu().numpy(), slack=out.slack[:R].cpu().numpy(),
                route=out.route[:R].cpu().numpy(), cost=out.cost[:R].cpu().numpy(),
                err=pol.last_error()), st.last_pass_incremental


def reasons(st):
    return st.last_fallback


def feed(st, p, prev_n, prev_done):
    """Snapshot p as the delta from the previous one: completions, then appends."""
    N = p.n_nodes
    if prev_n == 0:
        assert st.set_workflows(p.deadline_us) == nalar.NALAR_OK
        assert st.set_instances(p.inst_type, p.inst_load_us, p.inst_speed_permille) == nalar.NALAR_OK
    else:
        newly = np.flatnonzero((p.done[:prev_n] == 1) & (prev_done == 0)).astype(np.int32)
        assert st.complete(newly) == nalar.NALAR_OK
    e0, e1 = int(p.dep_off[prev_n]), int(p.dep_off[N])
    if N > prev_n:
        assert st.append(p.wf[prev_n:N], p.type[prev_n:N], p.est_us[prev_n:N], p.done[prev_n:N],
                         p.loc[prev_n:N], p.dep_off[prev_n:N + 1] - e0, p.dep_idx[e0:e1],
                         contiguous=bool(p.wf_contiguous)) == nalar.NALAR_OK
    return N, p.done[:N].copy()


# ------------------------------------------------------ map/reduce dynamic stream

_dyn = {}


def _dyn_state():
    if "it" not in _dyn:
        _dyn["it"] = wl.dynamic_stream(steps=100)
        _dyn["next"] = 0
        _dyn["pol"] = nalar.Policy()
        _dyn["st"] = nalar.Store(_dyn["pol"])
        _dyn["prev"] = (0, None)
        _dyn["inc"] = []
    return _dyn


@pytest.mark.parametrize("chunk", range(11))
def test_store_dynamic_stream_every_step(chunk):
    """Steps 0..100 of the evolving map/reduce graph fed to one store as
    deltas; every pass bit-exact against the oracle on the full snapshot, and
    every pass after the first incremental."""
    d = _dyn_state()
    lo, hi = (chunk * 10, chunk * 10 + 9) if chunk < 10 else (100, 100)
    assert d["next"] == lo, "chunks must run in order"
    pool = cf.ThreadPoolExecutor(max_workers=8)
    futs = []
    try:
        for step in range(lo, hi + 1):
            p = next(d["it"]).copy()
            d["next"] = step + 1
            d["prev"] = feed(d["st"], p, *d["prev"])
            say(f"[gpu] store dynamic step {step}: N={p.n_nodes}")
            g, inc = store_pass(d["pol"], d["st"], p)
            say(f"[gpu]   incremental={inc} fallback={d['st'].last_fallback} n_ready={g['n_ready']}")
            d["inc"].append(inc)
            futs.append((step, g, inc, pool.submit(oracle.run, p)))
        for step, g, inc, f in futs:
            assert_parity(g, f.result(), f"store dynamic step {step} (incremental={inc})")
    finally:
        pool.shutdown()
    if chunk == 10:
        d["st"].close()
        d["pol"].close()
        assert not d["inc"][0]
        full = [i for i, x in enumerate(d["inc"]) if not x and i > 0]
        assert len(full) <= 5, f"full passes at steps {full}"


# ------------------------------------------------------------- growing random DAGs

class Grower:
    """A random DAG grown in deltas.  Each step appends futures to random
    workflows (ids interleaved across workflows), each with 0..3 dependencies
    on earlier futures of its workflow, some on futures of the same call
    appended after it (a hidden topological order, then the call's ids
    shuffled), and now and then one with many dependencies; and marks a random
    set of futures done."""

    def __init__(self, seed, W=5, M=14, K=4, heavy=True):
        self.rng = np.random.default_rng(seed)
        self.W, self.M, self.K, self.heavy = W, M, K, heavy
        self.wf, self.type, self.est, self.done, self.loc = [], [], [], [], []
        self.deps = []
        self.now = int(self.rng.integers(0, 1000))
        self.deadline = (self.now + self.rng.integers(-200, 2000, W)).astype(np.int64)
        self.inst()

    def inst(self):
        r = self.rng
        self.inst_type = r.integers(0, self.K, self.M).astype(np.int32)
        self.inst_load = r.integers(0, 500, self.M).astype(np.int64)
        self.inst_speed = r.integers(1, 3000, self.M).astype(np.int32)

    def step(self, n_new):
        r = self.rng
        N0 = len(self.wf)
        hidden = []  # futures of this call in a hidden topological order
        for k in range(n_new):
            w = int(r.integers(0, self.W))
            pool = [v for v in range(N0) if self.wf[v] == w] + [N0 + j for j, (ww, _) in enumerate(hidden) if ww == w]
            nd = int(r.integers(0, 4))
            if self.heavy and pool and r.random() < 0.03:
                nd = int(r.integers(65, 140))
            deps = [int(x) for x in r.choice(pool, size=nd)] if pool and nd else []
            hidden.append((w, deps))
        perm = r.permutation(n_new)  # hidden position -> id offset
        rows = [None] * n_new
        for j, (w, deps) in enumerate(hidden):
            deps2 = [d if d < N0 else N0 + int(perm[d - N0]) for d in deps]
            rows[int(perm[j])] = (w, deps2)
        for w, deps in rows:
            self.wf.append(w)
            self.type.append(int(r.integers(0, self.K + 1)))
            e = int(r.integers(0, 60))
            self.est.append(0 if r.random() < 0.1 else e)
            self.done.append(1 if r.random() < 0.15 else 0)
            self.loc.append(int(r.integers(0, self.M)) if r.random() < 0.5 else -1)
            self.deps.append(deps)
        live = [v for v in range(N0) if self.done[v] == 0]
        if live:
            for v in r.choice(live, size=max(1, len(live) // 12), replace=False):
                self.done[int(v)] = 1

    def problem(self):
        N = len(self.wf)
        cnt = np.array([len(x) for x in self.deps], np.int64)
        off = np.zeros(N + 1, np.int64)
        np.cumsum(cnt, out=off[1:])
        idx = np.array([d for x in self.deps for d in x], np.int64)
        wf = np.array(self.wf, np.int32)
        return wl.Problem("grown", self.now, 150, wf, np.array(self.type, np.int32),
                          np.array(self.est, np.int64), np.array(self.done, np.uint8),
                          np.array(self.loc, np.int32), off.astype(np.int32), idx.astype(np.int32),
                          self.deadline.copy(), self.inst_type.copy(), self.inst_load.copy(),
                          self.inst_speed.copy(), wf_contiguous=bool(np.all(np.diff(wf) >= 0)))


@pytest.mark.parametrize("seed", range(6))
def test_store_incremental_random_growth(seed):
    """Growing random DAGs under every order and routing policy, with deadline
    and instance changes between some passes."""
    policies = [0, nalar.NALAR_ORDER_LPT, nalar.NALAR_ORDER_SRTF, nalar.NALAR_ROUTE_STATEFUL,
                nalar.NALAR_ROUTE_GREEDY, nalar.NALAR_ORDER_SRTF | nalar.NALAR_ROUTE_STATEFUL]
    bits = policies[seed % len(policies)]
    gr = Grower(7000 + seed)
    n_inc = 0
    with nalar.Policy() as pol:
        st = nalar.Store(pol)
        try:
            prev = (0, None)
            for step in range(14):
                gr.step(int(gr.rng.integers(20, 90)) if step else 120)
                if step % 5 == 4:
                    gr.deadline = gr.deadline + gr.rng.integers(-300, 300, gr.W)
                    assert st.set_workflows(gr.deadline) == nalar.NALAR_OK
                if step % 7 == 6:
                    gr.inst()
                    assert st.set_instances(gr.inst_type, gr.inst_load, gr.inst_speed) == nalar.NALAR_OK
                p = gr.problem()
                prev = feed(st, p, *prev)
                g, inc = store_pass(pol, st, p, bits)
                n_inc += inc
                say(f"[gpu] store growth seed {seed} step {step}: N={p.n_nodes} incremental={inc} "
                    f"fallback={st.last_fallback}")
                assert_parity(g, oracle.run(p, policy=bits), f"growth seed {seed} step {step}")
        finally:
            st.close()
    assert n_inc >= 10, n_inc


def test_store_incremental_and_full_agree():
    """One delta stream through two stores, one incremental and one with
    incremental passes off: equal results at every pass (and equal to the
    oracle), while the first store's passes after the first are incremental."""
    gr = Grower(7100, W=3, heavy=True)
    n_inc = 0
    with nalar.Policy() as pol_a, nalar.Policy() as pol_b:
        sa, sb = nalar.Store(pol_a), nalar.Store(pol_b)
        assert sb.set_incremental(False) == nalar.NALAR_OK
        try:
            pa = pb = (0, None)
            for step in range(10):
                gr.step(60)
                p = gr.problem()
                pa = feed(sa, p, *pa)
                pb = feed(sb, p, *pb)
                ga, ia = store_pass(pol_a, sa, p)
                gb, ib = store_pass(pol_b, sb, p)
                assert not ib
                if step == 0:
                    assert not ia
                n_inc += ia
                ref = oracle.run(p)
                assert_parity(ga, ref, f"incremental step {step}")
                assert_parity(gb, ref, f"full step {step}")
        finally:
            sa.close()
            sb.close()
    assert n_inc >= 8, n_inc


def test_store_incremental_errors():
    """Errors found by an incremental pass, with the codes of a full pass; the
    pass after a failure is a full one (and fails the same way while the bad
    futures stay)."""
    with nalar.Policy() as pol:
        # a cycle among appended futures (a dependency on a later future of the call)
        gr = Grower(7200, W=2, heavy=False)
        st = nalar.Store(pol)
        try:
            gr.step(80)
            p = gr.problem()
            prev = feed(st, p, 0, None)
            g, inc = store_pass(pol, st, p)
            assert_parity(g, oracle.run(p), "before the cycle")
            N = p.n_nodes
            w = int(p.wf[0])
            wf = np.full(2, w, np.int32)
            z = np.zeros(2, np.int32)
            assert st.append(wf, z, np.array([5, 6], np.int64), np.zeros(2, np.uint8), np.full(2, -1, np.int32),
                             np.array([0, 1, 2], np.int32), np.array([N + 1, N], np.int32)) == 0
            out = nalar.DeviceResult.alloc(N + 2)
            assert st.run_pass(out, p.now_us, p.migration_cost_us) == nalar.NALAR_ECYCLE
            assert st.last_pass_incremental
            assert st.run_pass(out, p.now_us, p.migration_cost_us) == nalar.NALAR_ECYCLE
            assert not st.last_pass_incremental
        finally:
            st.close()
        # a dependency on another workflow, then one out of range
        for bad_dep in ("other workflow", "out of range"):
            gr = Grower(7300, W=2, heavy=False)
            st = nalar.Store(pol)
            try:
                gr.step(60)
                p = gr.problem()
                feed(st, p, 0, None)
                g, _ = store_pass(pol, st, p)
                assert_parity(g, oracle.run(p), "before the bad dependency")
                N = p.n_nodes
                w = int(p.wf[0])
                if bad_dep == "other workflow":
                    other = int(np.flatnonzero(p.wf != w)[0])
                    dep = other
                else:
                    dep = N + 7
                assert st.append(np.array([w], np.int32), np.zeros(1, np.int32), np.array([3], np.int64),
                                 np.zeros(1, np.uint8), np.array([-1], np.int32), np.array([0, 1], np.int32),
                                 np.array([dep], np.int32)) == 0
                out = nalar.DeviceResult.alloc(N + 1)
                assert st.run_pass(out, p.now_us, p.migration_cost_us) == nalar.NALAR_EINVAL, bad_dep
                assert st.last_pass_incremental
            finally:
                st.close()
        # malformed appended offsets: the next pass fails
        st = nalar.Store(pol)
        try:
            gr = Grower(7400, W=2, heavy=False)
            gr.step(40)
            p = gr.problem()
            feed(st, p, 0, None)
            g, _ = store_pass(pol, st, p)
            assert_parity(g, oracle.run(p), "before the bad offsets")
            N = p.n_nodes
            assert st.append(np.zeros(1, np.int32), np.zeros(1, np.int32), np.array([3], np.int64),
                             np.zeros(1, np.uint8), np.array([-1], np.int32), np.array([1, 1], np.int32),
                             np.zeros(0, np.int32)) == 0
            out = nalar.DeviceResult.alloc(N + 1)
            assert st.run_pass(out, p.now_us, p.migration_cost_us) == nalar.NALAR_EINVAL
        finally:
            st.close()


def test_store_incremental_random_streams():
    """Two hundred small random streams (workflows, instances and types of
    random counts, heavy dependency lists in some, deadline and instance
    changes at random steps) under every order and routing policy: every pass,
    incremental or not, equals the oracle's pass over the snapshot."""
    pols = [0, nalar.NALAR_ORDER_LPT, nalar.NALAR_ORDER_SRTF, nalar.NALAR_ROUTE_STATEFUL,
            nalar.NALAR_ROUTE_GREEDY, nalar.NALAR_ORDER_SRTF | nalar.NALAR_ROUTE_STATEFUL,
            nalar.NALAR_ORDER_LPT | nalar.NALAR_ROUTE_GREEDY]
    n_pass = n_inc = 0
    for seed in range(200):
        rng = np.random.default_rng(90000 + seed)
        gr = Grower(50000 + seed, W=int(rng.integers(1, 12)), M=int(rng.integers(1, 40)),
                    K=int(rng.integers(1, 6)), heavy=bool(seed % 3))
        bits = pols[seed % len(pols)]
        with nalar.Policy() as pol:
            st = nalar.Store(pol)
            try:
                prev = (0, None)
                for step in range(int(rng.integers(5, 25))):
                    gr.step(int(rng.integers(1, 120)) if step else int(rng.integers(1, 200)))
                    if rng.random() < 0.15:
                        gr.deadline = gr.deadline + rng.integers(-300, 300, gr.W)
                        assert st.set_workflows(gr.deadline) == nalar.NALAR_OK
                    if rng.random() < 0.1:
                        gr.inst()
                        assert st.set_instances(gr.inst_type, gr.inst_load, gr.inst_speed) == nalar.NALAR_OK
                    p = gr.problem()
                    prev = feed(st, p, *prev)
                    g, inc = store_pass(pol, st, p, bits)
                    n_pass += 1
                    n_inc += inc
                    assert_parity(g, oracle.run(p, policy=bits), f"stream seed {seed} step {step} policy {bits}")
            finally:
                st.close()
    say(f"[gpu] random streams: {n_pass} passes, {n_inc} incremental")
    assert n_inc * 2 > n_pass, (n_inc, n_pass)
