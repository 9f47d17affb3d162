"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

The oracle is the reference every GPU result is compared with, so it is
checked here against things other than itself:

* hand-worked examples (tests/golden/, derivations written in each file);
* exhaustive path enumeration on small random DAGs (remaining work is the
  longest est'-weighted path, the remaining work ranked by SRTF, Section 6.2);
* a push-based replay of value deliveries for readiness (Section 4.3.1,
  property 3), a different formulation from the oracle's pull check;
* the optimality certificate of longest paths (edge inequality, equality on
  some consumer, sinks equal their own service time) on the full workloads;
* closed forms (chains, unit service times, the map/reduce shape);
* the routing special case with equal loads and speeds, and invariances;
* uniqueness of a sorted permutation under a total order;
* every validation and error rule of the boundary;
* the policy variants: LPT equals the slack order when deadlines are equal,
  its order certificate and a closed form; stateful routing against Python
  integer costs and against the default rule under prohibitive migration;
  greedy load-aware routing against prefix sums, round-robin and list
  scheduling closed forms, and monotonicity against the snapshot loads.
"""
import numpy as np
import pytest

import oracle
from golden_io import load as load_golden, names as golden_names
from paper_2601_05109_amd import workloads as wl


def wl_index(name):
    """The named workload's position in the table; its cases are seeded by it."""
    return list(wl.WORKLOADS).index(name)


INT64_MAX = np.iinfo(np.int64).max


# ---------------------------------------------------------------- helpers

def consumers(p):
    succ = [[] for _ in range(p.n_nodes)]
    for v in range(p.n_nodes):
        for e in range(p.dep_off[v], p.dep_off[v + 1]):
            succ[int(p.dep_idx[e])].append(v)
    return succ


def brute_force_rem(p):
    """Longest path by enumerating every directed path from each node."""
    N = p.n_nodes
    succ = consumers(p)
    w = [0 if p.done[v] else int(p.est_us[v]) for v in range(N)]
    out = []
    for v in range(N):
        best = 0
        stack = [(v, w[v])]
        while stack:
            u, s = stack.pop()
            best = max(best, s)
            for c in succ[u]:
                stack.append((c, s + w[c]))
        out.append(best)
    return np.array(out, np.int64)


def push_replay_ready(p):
    """Replay the pushes: each done future delivers its value once per
    dependency edge to its consumers; a not-done future that has received every
    delivery it waits for can run."""
    N = p.n_nodes
    need = np.diff(p.dep_off.astype(np.int64))
    got = np.zeros(N, np.int64)
    succ = consumers(p)
    for u in range(N):
        if p.done[u]:
            for c in succ[u]:
                got[c] += 1
    return {v for v in range(N) if not p.done[v] and got[v] == need[v]}


def assert_sorted_permutation(p, r):
    """order is the ready set, strictly increasing in (slack, wf, v): a sorted
    permutation under a total order is unique, so this pins the order."""
    keys = [(int(s), int(p.wf[v]), int(v)) for v, s in zip(r.order, r.slack)]
    assert all(a < b for a, b in zip(keys, keys[1:]))
    assert len(set(r.order.tolist())) == len(r.order)


def rem_certificate(p, rem):
    """Longest-path certificate: for every edge u->c, rem[u] >= est'[u] + rem[c];
    every node with consumers attains equality on one of them; a node without
    consumers has rem = est'.  By induction over a reverse topological order,
    these determine rem uniquely."""
    N = p.n_nodes
    e = np.where(p.done.astype(bool), 0, p.est_us).astype(np.int64)
    child = np.repeat(np.arange(N), np.diff(p.dep_off.astype(np.int64)))
    par = p.dep_idx.astype(np.int64)
    lhs = rem[par]
    rhs = e[par] + rem[child]
    assert np.all(lhs >= rhs), "edge inequality violated"
    best = np.full(N, -1, np.int64)
    np.maximum.at(best, par, rem[child])
    has = best >= 0
    assert np.all(rem[has] == e[has] + best[has]), "no tight consumer"
    assert np.all(rem[~has] == e[~has]), "sink base case"


# ---------------------------------------------------------------- golden

@pytest.mark.parametrize("name", golden_names())
def test_golden_examples(name):
    p, exp = load_golden(name)
    r = oracle.run(p)
    assert r.status == exp["status"][0]
    assert r.rem.tolist() == exp["rem"]
    assert r.order.tolist() == exp["order"]
    assert r.slack.tolist() == exp["slack"]
    assert r.route.tolist() == exp["route"]
    assert r.cost.tolist() == exp["cost"]


# ---------------------------------------------------------------- brute force

@pytest.mark.parametrize("seed", range(120))
def test_small_dags_against_brute_force(seed):
    rng = np.random.default_rng(seed)
    p = wl.random_dag(seed, n_nodes=int(rng.integers(1, 11)), n_workflows=int(rng.integers(1, 4)),
                      n_instances=int(rng.integers(0, 6)), n_types=int(rng.integers(1, 4)))
    r = oracle.run(p)
    assert r.status == oracle.OK
    np.testing.assert_array_equal(r.rem, brute_force_rem(p))
    assert set(r.order.tolist()) == push_replay_ready(p)
    assert_sorted_permutation(p, r)
    rem_certificate(p, r.rem)


def test_brute_force_catches_planted_mistakes():
    """The brute force and the certificate are sharp enough to reject a
    perturbed rem (one wrong entry anywhere)."""
    p = wl.random_dag(7, n_nodes=9, n_workflows=1, p_edge=0.5, zero_est=0.0, p_done=0.0)
    r = oracle.run(p)
    for v in range(p.n_nodes):
        bad = r.rem.copy()
        bad[v] += 1
        assert not np.array_equal(bad, brute_force_rem(p))
        with pytest.raises(AssertionError):
            rem_certificate(p, bad)


# ---------------------------------------------------------------- named workloads

@pytest.fixture(scope="module", params=list(wl.WORKLOADS))
def workload_run(request):
    p = wl.WORKLOADS[request.param]()
    return request.param, p, oracle.run(p)


def test_workload_certificate(workload_run):
    _, p, r = workload_run
    assert r.status == oracle.OK
    rem_certificate(p, r.rem)


def test_workload_order_and_ready(workload_run):
    c, p, r = workload_run
    assert_sorted_permutation(p, r)
    ready = np.zeros(p.n_nodes, bool)
    ready[r.order] = True
    # readiness by definition, vectorised: not done and no not-done parent
    child = np.repeat(np.arange(p.n_nodes), np.diff(p.dep_off.astype(np.int64)))
    blocked = np.zeros(p.n_nodes, bool)
    blocked[child[p.done[p.dep_idx] == 0]] = True
    np.testing.assert_array_equal(ready, (p.done == 0) & ~blocked)
    # stable-permutation property: the order equals a stable sort by
    # (slack, wf) of the ready ids listed in ascending id order
    ids = np.flatnonzero(ready)
    slack_of = dict(zip(r.order.tolist(), r.slack.tolist()))
    s = np.array([slack_of[v] for v in ids], np.int64)
    st = ids[np.lexsort((p.wf[ids], s))]    # lexsort is stable
    np.testing.assert_array_equal(st, r.order)


@pytest.mark.parametrize("name", ["tiny", "paper-scale"])
def test_windowed_ready_locality(name):
    """With the first 9 of 32 futures done and parents within the previous 8,
    every ready future has local index 9..16, and local index 9 is always ready."""
    p = wl.WORKLOADS[name]()
    r = oracle.run(p)
    local = r.order % 32
    assert local.min() >= 9 and local.max() <= 16
    assert set(np.flatnonzero(p.wf >= 0)[9::32].tolist()) <= set(r.order.tolist())


def test_mapreduce_closed_form():
    """Root done -> tools -> reduce: rem[reduce] = est[reduce],
    rem[tool] = est[tool] + est[reduce], rem[root] = max tool est + est[reduce];
    the ready set is exactly the tools, with slack deadline - now - rem."""
    p = wl.wide_mapreduce(W=8, fan=64)
    r = oracle.run(p)
    n = 66
    est = p.est_us.reshape(8, n)
    rem = r.rem.reshape(8, n)
    np.testing.assert_array_equal(rem[:, -1], est[:, -1])
    np.testing.assert_array_equal(rem[:, 1:-1], est[:, 1:-1] + est[:, -1:])
    np.testing.assert_array_equal(rem[:, 0], est[:, 1:-1].max(axis=1) + est[:, -1])
    tools = np.arange(8 * n).reshape(8, n)[:, 1:-1].reshape(-1)
    assert sorted(r.order.tolist()) == tools.tolist()
    w = p.wf[r.order]
    np.testing.assert_array_equal(r.slack, p.deadline_us[w] - p.now_us - r.rem[r.order])


def test_chain_suffix_sums():
    N = 50
    rng = np.random.default_rng(3)
    est = rng.integers(0, 10**6, N).astype(np.int64)
    done = (rng.random(N) < 0.3).astype(np.uint8)
    p = wl.Problem("chain", 0, 0, np.zeros(N, np.int32), np.zeros(N, np.int32), est, done,
                   -np.ones(N, np.int32), np.r_[0, 0, np.arange(1, N)].astype(np.int32),
                   np.arange(N - 1).astype(np.int32), np.array([10**9], np.int64),
                   np.zeros(0, np.int32), np.zeros(0, np.int64), np.zeros(0, np.int32), True)
    r = oracle.run(p)
    w = np.where(done == 1, 0, est)
    np.testing.assert_array_equal(r.rem, np.cumsum(w[::-1])[::-1])


def kahn_height(p):
    """Longest path length in edges, by peeling sinks level by level."""
    N = p.n_nodes
    succ = consumers(p)
    outdeg = np.array([len(s) for s in succ])
    par = [[] for _ in range(N)]
    for v in range(N):
        par[v] = [int(u) for u in p.dep_idx[p.dep_off[v]:p.dep_off[v + 1]]]
    h = np.zeros(N, np.int64)
    frontier = [v for v in range(N) if outdeg[v] == 0]
    level = 0
    while frontier:
        nxt = []
        for v in frontier:
            h[v] = level
            for u in par[v]:
                outdeg[u] -= 1
                if outdeg[u] == 0:
                    nxt.append(u)
        frontier = nxt
        level += 1
    return h


@pytest.mark.parametrize("seed", range(5))
def test_unit_service_time_is_height(seed):
    p = wl.deep_chains(seed=seed, W=4) if seed < 2 else wl.tiny(seed=seed)
    q = p.copy(est_us=np.ones(p.n_nodes, np.int64), done=np.zeros(p.n_nodes, np.uint8))
    r = oracle.run(q)
    np.testing.assert_array_equal(r.rem, kahn_height(q) + 1)


def test_relabelled_ids_give_relabelled_result():
    """Renaming node ids renames rem and order (ties within a workflow follow
    the new ids, so only the multiset of (slack, route, cost) per node is
    compared)."""
    p = wl.tiny()
    perm = np.random.default_rng(1).permutation(p.n_nodes)
    q = wl.relabel(p, perm)
    a, b = oracle.run(p), oracle.run(q)
    np.testing.assert_array_equal(b.rem[perm], a.rem)
    da = {int(perm[v]): (s, rt, c) for v, s, rt, c in zip(a.order, a.slack, a.route, a.cost)}
    db = {int(v): (s, rt, c) for v, s, rt, c in zip(b.order, b.slack, b.route, b.cost)}
    assert da == db


# ---------------------------------------------------------------- routing

def brute_route(p, v, mig=None):
    """Exhaustive minimum of (cost, index) over every instance of the
    future's type, in Python integers (no overflow, no rounding):
    cost = load + floor(est * 1000 / speed) + migration penalty unless the
    instance holds the future's state.  (INT64_MAX, -1) when none has the type."""
    mig = int(p.migration_cost_us) if mig is None else mig
    t, l, est = int(p.type[v]), int(p.loc[v]), int(p.est_us[v])
    cands = [(int(p.inst_load_us[i]) + (est * 1000) // int(p.inst_speed_permille[i])
              + (mig if (l >= 0 and l != i) else 0), i)
             for i in range(p.n_instances) if int(p.inst_type[i]) == t]
    if not cands:
        return INT64_MAX, -1
    return min(cands)


def assert_routes_exhaustive(p, r):
    for k, v in enumerate(r.order.tolist()):
        c, i = brute_route(p, v)
        assert (int(r.cost[k]), int(r.route[k])) == (c, i), (p.name, v)


def wide_range(p, seed):
    """The same graph with estimates, loads, speeds and migration cost drawn
    over the whole range the boundary accepts (est up to 2^40, load and
    migration up to 2^60, speed up to 2^31 - 1), loads often tied."""
    rng = np.random.default_rng(seed)
    N, M = p.n_nodes, p.n_instances
    est = rng.integers(0, 1 << 40, N, dtype=np.int64, endpoint=True)
    est[rng.random(N) < 0.2] = 0
    load = rng.choice([0, 7, 1 << 60, int(rng.integers(0, 1 << 60))], M).astype(np.int64)
    speed = rng.choice([1, 1000, (1 << 31) - 1, int(rng.integers(1, 1 << 31))], M).astype(np.int32)
    return p.copy(est_us=est, inst_load_us=load, inst_speed_permille=speed,
                  migration_cost_us=int(rng.choice([0, 200_000, 1 << 60])))


@pytest.mark.parametrize("name", ["tiny", "paper-scale"])
def test_route_exhaustive_workloads(name):
    """Every ready future of the tiny and paper-scale snapshots is routed to
    the exhaustive big-integer minimum of (cost, index)."""
    p = wl.WORKLOADS[name]()
    r = oracle.run(p)
    assert r.status == oracle.OK and r.n_ready > 0
    assert_routes_exhaustive(p, r)


@pytest.mark.parametrize("seed", range(150))
def test_route_exhaustive_random(seed):
    """Small DAGs with unequal loads and speeds, migration penalties, state on
    instances of other types, ties and futures of types no instance has; every
    fifth over the full value range of the boundary."""
    rng = np.random.default_rng(1000 + seed)
    p = wl.random_dag(500 + seed, n_nodes=int(rng.integers(1, 40)), n_workflows=int(rng.integers(1, 4)),
                      n_instances=int(rng.integers(0, 12)), n_types=int(rng.integers(1, 5)),
                      load_max=int(rng.choice([3, 100, 10**6])), speed_hi=int(rng.choice([2, 3000])))
    if seed % 5 == 0 and p.n_instances > 0:
        p = wide_range(p, seed)
    r = oracle.run(p)
    assert r.status == oracle.OK
    assert_routes_exhaustive(p, r)


def test_route_exhaustive_catches_planted_mistakes():
    """The exhaustive pin rejects a swapped load and service term, a penalty
    charged on the state's own instance, and ties to the higher index."""
    p = wl.tiny()
    r = oracle.run(p)
    bad_swap = r.cost.copy()
    v0 = int(r.order[0])
    c, i = brute_route(p, v0)
    for k, v in enumerate(r.order.tolist()):
        l = int(p.loc[v])
        if l >= 0 and int(p.inst_type[l]) == int(p.type[v]):
            bad = r.cost.copy()
            bad[k] += int(p.migration_cost_us)
            with pytest.raises(AssertionError):
                assert_routes_exhaustive(p, oracle.OracleResult(0, r.n_ready, r.rem, r.order, r.slack, r.route, bad))
            break
    bad_swap[0] = int(p.est_us[v0]) + int(p.inst_load_us[i]) * 1000 // int(p.inst_speed_permille[i])
    with pytest.raises(AssertionError):
        assert_routes_exhaustive(p, oracle.OracleResult(0, r.n_ready, r.rem, r.order, r.slack, r.route, bad_swap))


def test_route_equal_loads_closed_form():
    """Equal loads and speed 1000 everywhere: the future goes where its state
    is when that instance has its type, otherwise to the lowest-index instance
    of its type, and to -1 when there is none."""
    p = wl.tiny()
    M = p.n_instances
    q = p.copy(inst_load_us=np.full(M, 777, np.int64), inst_speed_permille=np.full(M, 1000, np.int32))
    r = oracle.run(q)
    for v, rt in zip(r.order.tolist(), r.route.tolist()):
        t, l = int(q.type[v]), int(q.loc[v])
        same = np.flatnonzero(q.inst_type == t)
        if same.size == 0:
            assert rt == -1
        elif l >= 0 and q.inst_type[l] == t:
            assert rt == l
        else:
            assert rt == same[0]


def test_route_invariant_to_common_load_shift():
    p = wl.tiny()
    r0 = oracle.run(p)
    r1 = oracle.run(p.copy(inst_load_us=p.inst_load_us + 123_456))
    np.testing.assert_array_equal(r0.route, r1.route)
    ok = r0.route >= 0
    np.testing.assert_array_equal(r1.cost[ok], r0.cost[ok] + 123_456)


def test_route_prohibitive_migration_keeps_state_local():
    p = wl.tiny()
    r = oracle.run(p.copy(migration_cost_us=1 << 60))
    for v, rt in zip(r.order.tolist(), r.route.tolist()):
        l = int(p.loc[v])
        if l >= 0 and p.inst_type[l] == p.type[v]:
            assert rt == l


def test_route_no_instances():
    p = wl.tiny()
    q = p.copy(inst_type=np.zeros(0, np.int32), inst_load_us=np.zeros(0, np.int64),
               inst_speed_permille=np.zeros(0, np.int32), loc=np.full(p.n_nodes, -1, np.int32))
    r = oracle.run(q)
    assert r.status == oracle.OK
    assert np.all(r.route == -1) and np.all(r.cost == INT64_MAX)


# ---------------------------------------------------------------- policy variants

LPT, STATEFUL = oracle.POLICY_LPT, oracle.POLICY_STATEFUL


def test_lpt_equals_srtf_when_deadlines_are_equal():
    """With one deadline for every workflow, slack = D - now - rem, so the
    slack order (pinned above) and the longest-remaining-work order (the LPT
    policy, Section 6.2) coincide, tie-breaks included."""
    for p in (wl.tiny(), wl.paper_scale(), wl.random_dag(7, n_nodes=300, n_workflows=5)):
        q = p.copy(deadline_us=np.full(p.n_workflows, p.now_us + 5_000_000, np.int64))
        a, b = oracle.run(q), oracle.run(q, policy=LPT)
        for f in ("order", "slack", "route", "cost", "rem"):
            np.testing.assert_array_equal(getattr(a, f), getattr(b, f))


@pytest.mark.parametrize("name", ["tiny", "paper-scale", "wide-mapreduce"])
def test_lpt_order_certificate(name):
    """The LPT order is a permutation of the ready set (the same set as the
    default pass) strictly increasing in (-rem, wf, v): unique under a total
    order; slack, route and cost are those of the default pass, permuted."""
    p = wl.WORKLOADS[name]()
    a, b = oracle.run(p), oracle.run(p, policy=LPT)
    assert b.n_ready == a.n_ready
    assert sorted(b.order.tolist()) == sorted(a.order.tolist())
    keys = [(-int(b.rem[v]), int(p.wf[v]), int(v)) for v in b.order.tolist()]
    assert all(x < y for x, y in zip(keys, keys[1:]))
    by_v = {int(v): i for i, v in enumerate(a.order.tolist())}
    idx = np.array([by_v[int(v)] for v in b.order.tolist()], np.int64)
    for f in ("slack", "route", "cost"):
        np.testing.assert_array_equal(getattr(b, f), getattr(a, f)[idx])


def test_lpt_independent_futures_closed_form():
    """Independent futures (no dependencies, none done): rem = est, so LPT lists
    them by est descending, ties by workflow then id."""
    N, W = 40, 3
    rng = np.random.default_rng(5)
    p = wl.random_dag(3, n_nodes=N, n_workflows=W, p_edge=0.0)
    p = p.copy(done=np.zeros(N, np.uint8), est_us=rng.integers(0, 6, N).astype(np.int64))
    r = oracle.run(p, policy=LPT)
    want = sorted(range(N), key=lambda v: (-int(p.est_us[v]), int(p.wf[v]), v))
    assert r.order.tolist() == want


def test_stateful_routing_pins():
    """Futures whose state lives on an instance of their own type run there at
    that instance's cost (load + floor(est*1000/speed), computed here with
    Python integers); every other future is routed as by the default rule.
    Equivalently, the stateful choice is what the default rule picks when
    migration is prohibitively expensive."""
    p = wl.paper_scale()
    a = oracle.run(p)
    s = oracle.run(p, policy=STATEFUL)
    h = oracle.run(p.copy(migration_cost_us=1 << 60))
    assert s.order.tolist() == a.order.tolist()
    pinned = 0
    for k, v in enumerate(s.order.tolist()):
        l, t = int(p.loc[v]), int(p.type[v])
        if l >= 0 and int(p.inst_type[l]) == t:
            pinned += 1
            assert s.route[k] == l == h.route[k]
            assert s.cost[k] == int(p.inst_load_us[l]) + int(p.est_us[v]) * 1000 // int(p.inst_speed_permille[l])
            assert s.cost[k] == h.cost[k]
        else:
            assert s.route[k] == a.route[k] and s.cost[k] == a.cost[k]
    assert pinned > 500


def test_stateful_without_state_is_default():
    p = wl.tiny()
    q = p.copy(loc=np.full(p.n_nodes, -1, np.int32))
    a, s = oracle.run(q), oracle.run(q, policy=STATEFUL | LPT)
    b = oracle.run(q, policy=LPT)
    for f in ("order", "slack", "route", "cost"):
        np.testing.assert_array_equal(getattr(s, f), getattr(b, f))
    np.testing.assert_array_equal(np.sort(a.route), np.sort(s.route))


def test_unknown_policy_bits_rejected():
    assert oracle.run(wl.tiny(), policy=64).status == oracle.EINVAL
    assert oracle.run(wl.tiny(), policy=LPT | oracle.POLICY_SRTF).status == oracle.EINVAL


SRTF = oracle.POLICY_SRTF


@pytest.mark.parametrize("name", ["tiny", "paper-scale", "deep-chains", "wide-mapreduce"])
def test_srtf_order_certificate(name):
    """SRTF (least remaining work first, Section 6.2): the ready set of the
    default pass, strictly increasing in (rem, wf, v), which is unique under
    that total order; slack, route and cost are the default pass's, permuted."""
    p = wl.WORKLOADS[name]()
    a, b = oracle.run(p), oracle.run(p, policy=SRTF)
    assert b.n_ready == a.n_ready
    assert sorted(b.order.tolist()) == sorted(a.order.tolist())
    keys = [(int(b.rem[v]), int(p.wf[v]), int(v)) for v in b.order.tolist()]
    assert all(x < y for x, y in zip(keys, keys[1:]))
    by_v = {int(v): i for i, v in enumerate(a.order.tolist())}
    idx = np.array([by_v[int(v)] for v in b.order.tolist()], np.int64)
    for f in ("slack", "route", "cost"):
        np.testing.assert_array_equal(getattr(b, f), getattr(a, f)[idx])


def test_srtf_is_lpt_reversed_for_distinct_work():
    """With pairwise distinct remaining work, least-remaining-first is exactly
    longest-remaining-first read backwards.  Estimates are distinct powers of
    two, so each rem (a sum over the set of futures on one path) is distinct:
    two start nodes with the same path set would reach each other."""
    rng = np.random.default_rng(3)
    p = wl.random_dag(21, n_nodes=40, n_workflows=4, p_edge=0.1)
    p = p.copy(est_us=(np.int64(1) << rng.permutation(40).astype(np.int64)), done=np.zeros(40, np.uint8))
    a, b = oracle.run(p, policy=SRTF), oracle.run(p, policy=LPT)
    ready_rem = a.rem[a.order]
    assert len(set(ready_rem.tolist())) == len(ready_rem)
    assert a.order.tolist() == b.order.tolist()[::-1]


def test_srtf_independent_futures_closed_form():
    """Independent futures, none done: rem = est, so SRTF lists them by est
    ascending, ties by workflow then id."""
    N, W = 40, 3
    rng = np.random.default_rng(6)
    p = wl.random_dag(4, n_nodes=N, n_workflows=W, p_edge=0.0)
    p = p.copy(done=np.zeros(N, np.uint8), est_us=rng.integers(0, 6, N).astype(np.int64))
    r = oracle.run(p, policy=SRTF)
    assert r.order.tolist() == sorted(range(N), key=lambda v: (int(p.est_us[v]), int(p.wf[v]), v))


WEIGHTED = oracle.POLICY_WEIGHTED


def quota_dispatch(p, order, weights, skip=()):
    """A weighted dispatcher written as a stateful quota walk (a different
    formulation from the oracle's modular arithmetic): per type, a pointer to
    the current instance and its remaining quota; a future takes the current
    instance and uses one unit of its quota; an exhausted quota moves the
    pointer to the next instance of the type with a positive weight (cyclic,
    by index) and refills it with that instance's weight.  Futures in ``skip``
    are passed over.  Returns {future: instance} for weighted types only."""
    state = {}
    out = {}
    for v in order:
        if v in skip:
            continue
        t = int(p.type[v])
        insts = [i for i in range(p.n_instances) if int(p.inst_type[i]) == t and int(weights[i]) > 0]
        if not insts:
            continue
        ptr, quota = state.get(t, (0, int(weights[insts[0]])))
        while quota == 0:
            ptr = (ptr + 1) % len(insts)
            quota = int(weights[insts[ptr]])
        out[v] = insts[ptr]
        state[t] = (ptr, quota - 1)
    return out


@pytest.mark.parametrize("name", ["tiny", "paper-scale"])
def test_weighted_against_quota_walk(name):
    """Weighted routing (Table 2's route by a list of instances and weights):
    every weighted future goes where the quota walk sends it, at the
    exhaustive cost of that instance; unweighted types keep the default route;
    the order is untouched."""
    p = wl.WORKLOADS[name]()
    rng = np.random.default_rng(40 + wl_index(name))
    w = rng.integers(0, 5, p.n_instances).astype(np.uint32)
    w[p.inst_type == 1] = 0            # one type without weights: default routing
    a, r = oracle.run(p), oracle.run(p, policy=WEIGHTED, weights=w)
    assert r.status == oracle.OK
    for f in ("order", "slack", "rem"):
        np.testing.assert_array_equal(getattr(a, f), getattr(r, f))
    want = quota_dispatch(p, r.order.tolist(), w)
    assert len(want) > r.n_ready // 4
    mig = int(p.migration_cost_us)
    for k, v in enumerate(r.order.tolist()):
        if v in want:
            i = want[v]
            assert int(r.route[k]) == i
            l = int(p.loc[v])
            assert int(r.cost[k]) == (int(p.inst_load_us[i]) + int(p.est_us[v]) * 1000 // int(p.inst_speed_permille[i])
                                      + (mig if l >= 0 and l != i else 0))
        else:
            assert (int(r.route[k]), int(r.cost[k])) == (int(a.route[k]), int(a.cost[k]))


def test_weighted_unit_weights_round_robin():
    """Weight one on every instance of a single type: plain round-robin in
    index order, the k-th future (in output order) on instance k mod m."""
    m, n = 5, 23
    p = _one_type_problem(m, [0] * m, [1000] * m, [10] * n)
    r = oracle.run(p, policy=WEIGHTED, weights=np.ones(m, np.uint32))
    np.testing.assert_array_equal(r.route, np.arange(n) % m)


def test_weighted_whole_periods_are_proportional():
    """After a whole number of periods (futures = a multiple of the total
    weight) every instance has received exactly its weight times the number
    of periods; instances of weight zero receive nothing."""
    w = np.array([3, 0, 1, 4, 2], np.uint32)
    n = 4 * int(w.sum())
    p = _one_type_problem(len(w), [9] * len(w), [1000] * len(w), [10] * n)
    r = oracle.run(p, policy=WEIGHTED, weights=w)
    np.testing.assert_array_equal(np.bincount(r.route, minlength=len(w)), 4 * w)


def test_weighted_rules():
    """Weights above 2^20, missing weights and weighted with greedy routing are
    EINVAL; all-zero weights give the default routing; a stateful pin keeps
    its instance and takes no place in its type's sequence."""
    p = wl.tiny()
    M = p.n_instances
    assert oracle.run(p, policy=WEIGHTED).status == oracle.EINVAL
    big = np.ones(M, np.uint32)
    big[2] = (1 << 20) + 1
    assert oracle.run(p, policy=WEIGHTED, weights=big).status == oracle.EINVAL
    assert oracle.run(p, policy=WEIGHTED | GREEDY, weights=np.ones(M, np.uint32)).status == oracle.EINVAL
    a, z = oracle.run(p), oracle.run(p, policy=WEIGHTED, weights=np.zeros(M, np.uint32))
    for f in ("order", "route", "cost"):
        np.testing.assert_array_equal(getattr(a, f), getattr(z, f))
    w = np.arange(1, M + 1).astype(np.uint32) % 3
    s = oracle.run(p, policy=WEIGHTED | STATEFUL, weights=w)
    pinned = {int(v) for v in s.order.tolist()
              if int(p.loc[v]) >= 0 and int(p.inst_type[int(p.loc[v])]) == int(p.type[v])}
    assert pinned
    want = quota_dispatch(p, s.order.tolist(), w, skip=pinned)
    for k, v in enumerate(s.order.tolist()):
        if v in pinned:
            assert int(s.route[k]) == int(p.loc[v])
        elif v in want:
            assert int(s.route[k]) == want[v]


GREEDY = oracle.POLICY_GREEDY


def _one_type_problem(n_inst, loads, speeds, est, loc=None, mig=200_000, deadline_spread=True):
    """Independent futures (no dependencies, none done) of one type in one
    workflow each, against n_inst instances of that type."""
    N = len(est)
    rng = np.random.default_rng(N)
    dl = 1_000_000 + (rng.permutation(N) * 1000 if deadline_spread else np.zeros(N, np.int64))
    now = 1_000
    return wl.Problem("one-type", now, mig, np.arange(N, dtype=np.int32), np.zeros(N, np.int32),
                      np.asarray(est, np.int64), np.zeros(N, np.uint8),
                      np.full(N, -1, np.int32) if loc is None else np.asarray(loc, np.int32),
                      np.zeros(N + 1, np.int32), np.zeros(0, np.int32),
                      (now + dl).astype(np.int64), np.zeros(n_inst, np.int32),
                      np.asarray(loads, np.int64), np.asarray(speeds, np.int32), wf_contiguous=True)


def test_greedy_single_instance_prefix_sums():
    """One instance: every future goes there and waits for all before it in the
    output order, so its cost is the initial load plus the prefix sum of
    service times (est * 1000 // speed) up to and including itself."""
    rng = np.random.default_rng(1)
    est = rng.integers(0, 10**6, 50)
    p = _one_type_problem(1, [12345], [750], est)
    r = oracle.run(p, policy=GREEDY)
    svc = np.array([int(est[v]) * 1000 // 750 for v in r.order.tolist()], np.int64)
    assert np.all(r.route == 0)
    np.testing.assert_array_equal(r.cost, 12345 + np.cumsum(svc))


def test_greedy_identical_instances_round_robin():
    """Identical instances and identical futures: list scheduling deals them
    out in index order (ties go to the lowest index): route k mod m, and the
    k-th future waits k // m service times before its own."""
    m, n = 3, 20
    p = _one_type_problem(m, [500] * m, [1000] * m, [40] * n)
    r = oracle.run(p, policy=GREEDY)
    k = np.arange(n)
    np.testing.assert_array_equal(r.route, k % m)
    np.testing.assert_array_equal(r.cost, 500 + (k // m + 1) * 40)


@pytest.mark.parametrize("name", ["tiny", "paper-scale"])
def test_greedy_invariants(name):
    """Loads only grow, so no future costs less than under the snapshot loads;
    the first future of each type in the order is routed exactly as by the
    default rule; order and slack are untouched."""
    p = wl.WORKLOADS[name]()
    a, g = oracle.run(p), oracle.run(p, policy=GREEDY)
    for f in ("order", "slack", "rem"):
        np.testing.assert_array_equal(getattr(a, f), getattr(g, f))
    ok = a.route >= 0
    assert np.all((g.route >= 0) == ok)
    assert np.all(g.cost[ok] >= a.cost[ok])
    seen = set()
    for k, v in enumerate(a.order.tolist()):
        t = int(p.type[v])
        if t not in seen:
            seen.add(t)
            assert g.route[k] == a.route[k] and g.cost[k] == a.cost[k]


def test_greedy_balances_identical_instances():
    """List scheduling of equal jobs on identical machines: the final loads
    differ by at most one service time."""
    m, n = 4, 37
    p = _one_type_problem(m, [0] * m, [1000] * m, [25] * n)
    r = oracle.run(p, policy=GREEDY)
    counts = np.bincount(r.route, minlength=m)
    assert counts.max() - counts.min() <= 1


def test_greedy_load_overflow_is_erange():
    # each future adds 2^40 * 1000 (about 2^50) to the one instance's load,
    # which starts at 2^60: the 3072nd addition or so passes 2^62
    p = _one_type_problem(1, [1 << 60], [1], [1 << 40] * 3200)
    assert oracle.run(p).status == oracle.OK
    assert oracle.run(p, policy=GREEDY).status == oracle.ERANGE


@pytest.mark.parametrize("name", ["tiny", "paper-scale"])
def test_priority_levels_partition_the_order(name):
    """set_priority levels per workflow: the order is the default order split
    stably by level, highest level first; slack, route and cost travel with
    their futures; equal levels change nothing."""
    p = wl.WORKLOADS[name]()
    rng = np.random.default_rng(wl_index(name))
    base = oracle.run(p)
    flat = oracle.run(p, priority=np.full(p.n_workflows, 7, np.uint8))
    for f in ("order", "slack", "route", "cost", "rem"):
        np.testing.assert_array_equal(getattr(base, f), getattr(flat, f))
    for bits in (0, LPT):
        pr = rng.integers(0, 16, p.n_workflows).astype(np.uint8)
        a, b = oracle.run(p, policy=bits), oracle.run(p, policy=bits, priority=pr)
        lv = pr[p.wf[a.order]]
        want = np.concatenate([a.order[lv == x] for x in range(15, -1, -1)])
        np.testing.assert_array_equal(b.order, want)
        pos = {int(v): i for i, v in enumerate(a.order.tolist())}
        idx = np.array([pos[int(v)] for v in b.order.tolist()], np.int64)
        for f in ("slack", "route", "cost"):
            np.testing.assert_array_equal(getattr(b, f), getattr(a, f)[idx])


def test_priority_level_and_key_rules():
    """A level above 15 is EINVAL; any key is ordered by the plain rule
    (level first, then key, workflow, id), also keys far outside any clock
    range: slacks near +-2^61 split by level exactly as small ones do."""
    p = wl.tiny()
    pr = np.zeros(p.n_workflows, np.uint8)
    pr[3] = 16
    assert oracle.run(p, priority=pr).status == oracle.EINVAL
    rng = np.random.default_rng(11)
    dl = p.now_us + rng.choice([-(1 << 61), (1 << 61) - (1 << 40), 0, 1 << 58], p.n_workflows)
    far = p.copy(deadline_us=dl.astype(np.int64))
    base = oracle.run(far)
    assert base.status == oracle.OK
    assert base.slack.min() < -(1 << 60) and base.slack.max() > (1 << 60)
    for bits in (0, LPT, oracle.POLICY_SRTF):
        pr = rng.integers(0, 16, p.n_workflows).astype(np.uint8)
        a, b = oracle.run(far, policy=bits), oracle.run(far, policy=bits, priority=pr)
        assert b.status == oracle.OK
        lv = pr[p.wf[a.order]]
        want = np.concatenate([a.order[lv == x] for x in range(15, -1, -1)])
        np.testing.assert_array_equal(b.order, want)


# ---------------------------------------------------------------- degenerate

def _single(est=5, done=0):
    return wl.Problem("one", 10, 7, np.zeros(1, np.int32), np.zeros(1, np.int32),
                      np.array([est], np.int64), np.array([done], np.uint8), np.array([0], np.int32),
                      np.array([0, 0], np.int32), np.zeros(0, np.int32), np.array([20], np.int64),
                      np.array([0], np.int32), np.array([3], np.int64), np.array([1000], np.int32), True)


def test_single_node():
    r = oracle.run(_single())
    assert r.status == 0 and r.order.tolist() == [0] and r.slack.tolist() == [5]
    assert r.route.tolist() == [0] and r.cost.tolist() == [8] and r.rem.tolist() == [5]


def test_empty_problem():
    p = _single()
    q = p.copy(wf=np.zeros(0, np.int32), type=np.zeros(0, np.int32), est_us=np.zeros(0, np.int64),
               done=np.zeros(0, np.uint8), loc=np.zeros(0, np.int32), dep_off=np.array([0], np.int32))
    r = oracle.run(q)
    assert r.status == 0 and r.n_ready == 0


def test_all_done():
    p = wl.tiny()
    r = oracle.run(p.copy(done=np.ones(p.n_nodes, np.uint8)))
    assert r.status == 0 and r.n_ready == 0
    assert np.all(r.rem == 0)


def test_no_edges_everything_ready():
    p = wl.tiny()
    N = p.n_nodes
    q = p.copy(dep_off=np.zeros(N + 1, np.int32), dep_idx=np.zeros(0, np.int32),
               done=np.zeros(N, np.uint8))
    r = oracle.run(q)
    assert r.n_ready == N
    np.testing.assert_array_equal(r.rem, q.est_us)


# ---------------------------------------------------------------- errors

def _bad(field, idx, value, base=None):
    p = (base or wl.tiny()).copy()
    getattr(p, field)[idx] = value
    return p


@pytest.mark.parametrize("case", [
    ("wf", 5, -1), ("wf", 5, 64), ("type", 3, -1), ("loc", 7, -2), ("loc", 7, 16),
    ("est_us", 9, -1), ("est_us", 9, (1 << 40) + 1), ("done", 4, 2),
    ("dep_idx", 10, -1), ("dep_idx", 10, 2048), ("dep_idx", 10, 40),   # 40 lies in workflow 1
    ("dep_off", 0, 1), ("dep_off", 2048, 1), ("inst_type", 0, -1),
    ("inst_speed_permille", 2, 0), ("inst_load_us", 1, -1), ("inst_load_us", 1, (1 << 60) + 1),
    ("deadline_us", 3, wl.NOW_US + (1 << 61) + 1),
])
def test_einval_rules(case):
    assert oracle.run(_bad(*case)).status == oracle.EINVAL


def test_einval_decreasing_offsets():
    p = wl.tiny().copy()
    p.dep_off[100], p.dep_off[101] = p.dep_off[101], p.dep_off[100]
    if p.dep_off[100] == p.dep_off[101]:
        pytest.skip("equal offsets")
    assert oracle.run(p).status == oracle.EINVAL


@pytest.mark.parametrize("ov", [dict(M=1025), dict(N=-1), dict(now=(1 << 61) + 1),
                                dict(mig=-1), dict(mig=(1 << 60) + 1), dict(E=5),
                                dict(wf=None), dict(dep_idx=None), dict(deadline_us=None),
                                dict(inst_speed_permille=None)])
def test_einval_scalars_and_nulls(ov):
    assert oracle.run(wl.tiny(), override=ov).status == oracle.EINVAL


def test_ecycle_self_loop_and_cycle():
    p = wl.tiny().copy()
    v = 12
    p.dep_idx[p.dep_off[v]] = v          # self-dependency
    assert oracle.run(p).status == oracle.ECYCLE
    # 0 -> 1 -> 2 -> 0 (node 0 depends on 2, node 1 on 0, node 2 on 1)
    N = 3
    c = wl.Problem("cyc", 0, 0, np.zeros(N, np.int32), np.zeros(N, np.int32), np.ones(N, np.int64),
                   np.zeros(N, np.uint8), -np.ones(N, np.int32), np.array([0, 1, 2, 3], np.int32),
                   np.array([2, 0, 1], np.int32), np.array([100], np.int64), np.zeros(0, np.int32),
                   np.zeros(0, np.int64), np.zeros(0, np.int32), True)
    assert oracle.run(c).status == oracle.ECYCLE


def test_erange_and_precedence():
    N = 4100
    # a chain of 4100 futures of 2^40 us each: rem reaches ~2^52, fine
    chain = lambda est, n: wl.Problem(
        "chain", 0, 0, np.zeros(n, np.int32), np.zeros(n, np.int32), np.full(n, est, np.int64),
        np.zeros(n, np.uint8), -np.ones(n, np.int32), np.r_[0, 0, np.arange(1, n)].astype(np.int32),
        np.arange(n - 1).astype(np.int32), np.array([0], np.int64), np.zeros(0, np.int32),
        np.zeros(0, np.int64), np.zeros(0, np.int32), True)
    assert oracle.run(chain(1 << 40, N)).status == oracle.OK
    # 2^22 + 1 futures of 2^40 us exceed 2^62
    big = chain(1 << 40, (1 << 22) + 1)
    assert oracle.run(big).status == oracle.ERANGE
    # a cycle takes precedence over an overflow
    cyc = big.copy()
    cyc.dep_idx[0] = 5       # node 1 depends on node 5, which descends from it
    assert oracle.run(cyc).status == oracle.ECYCLE
    # invalid input takes precedence over both
    inv = cyc.copy()
    inv.type[3] = -4
    assert oracle.run(inv).status == oracle.EINVAL
