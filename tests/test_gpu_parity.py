"""GPU parity: the HIP pass through the C ABI versus the CPU oracle.

Every comparison is bit-exact (all arithmetic is integer): remaining critical
path of every future, the ready order, slack, route and cost, and the return
code.  Cases: hand-worked fixtures, small random DAGs (contiguous and shuffled
ids, many instances/types, duplicate dependencies), the tiny / paper-scale /
deep-chain / map-reduce workloads, relabelled ids (the library groups futures by
workflow itself), the HBM sweep path forced on (with topological ids the
ordered chunk pass, with shuffled ids or NALAR_FORCE_LEVEL_SWEEP the level
sweep), workflows of several chunks with chains and heavy futures inside a
chunk, every error rule, repeated passes, scratch reuse across sizes, and
every step of the dynamic stream.
"""
import concurrent.futures as cf
import os
import sys

import numpy as np
import pytest

import oracle
from golden_io import load as load_golden, names as golden_names
from paper_2601_05109_amd import workloads as wl
from test_oracle_pins import wl_index

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover - collected on CPU hosts too
    pytest.skip("no GPU", allow_module_level=True)

from paper_2601_05109_amd import nalar  # noqa: E402


def say(msg):
    sys.stdout.write(msg + "\n")
    sys.stdout.flush()


@pytest.fixture(scope="module")
def policy():
    with nalar.Policy() as p:
        yield p


@pytest.fixture(scope="module")
def policy_hbm():
    with nalar.Policy(flags=nalar.NALAR_FORCE_GLOBAL_SWEEP) as p:
        yield p


@pytest.fixture(scope="module")
def policy_hbm_levels():
    """Every workflow in HBM, swept level by level (never the ordered chunk pass)."""
    with nalar.Policy(flags=nalar.NALAR_FORCE_GLOBAL_SWEEP | nalar.NALAR_FORCE_LEVEL_SWEEP) as p:
        yield p


@pytest.fixture(scope="module")
def policy_tiled():
    with nalar.Policy(flags=nalar.NALAR_FORCE_TILED_SORT) as p:
        yield p


def seeded_weights(p):
    """Routing weights for NALAR_ROUTE_WEIGHTED cases: 0..4 per instance,
    seeded by the problem's size, with one type left unweighted."""
    w = np.random.default_rng(p.n_instances * 7 + p.n_nodes).integers(0, 5, p.n_instances).astype(np.uint32)
    if p.n_instances:
        w[p.inst_type == p.inst_type[0]] = 0
    return w


def gpu_run(pol, p, flags=None, policy=0, priority=None, weights=None):
    dp = nalar.DeviceProblem.from_host(p)
    out = nalar.DeviceResult.alloc(dp.n_nodes)
    pr = None if priority is None else torch.from_numpy(np.ascontiguousarray(priority, np.uint8)).cuda()
    wt = None if weights is None else torch.from_numpy(np.ascontiguousarray(weights, np.uint32).view(np.int32)).cuda()
    cp = dp.c_struct(flags, policy, pr, wt)
    rc = pol.run_pass(dp, out, raw=cp)
    torch.cuda.synchronize()
    R = out.n_ready
    N = dp.n_nodes
    return dict(status=rc, n_ready=R, rem=out.rem[:N].cpu().numpy(),
                order=out.order[:R].cpu().numpy(), slack=out.slack[:R].cpu().numpy(),
                route=out.route[:R].cpu().numpy(), cost=out.cost[:R].cpu().numpy(),
                err=pol.last_error())


def assert_parity(g, o, label=""):
    assert g["status"] == o.status, f"{label}: status gpu={g['status']} ({g['err']}) oracle={o.status}"
    if o.status != oracle.OK:
        return
    assert g["n_ready"] == o.n_ready, f"{label}: n_ready {g['n_ready']} vs {o.n_ready}"
    for f, ref in (("rem", o.rem), ("order", o.order), ("slack", o.slack), ("route", o.route),
                   ("cost", o.cost)):
        got = g[f]
        if not np.array_equal(got, ref):
            bad = np.flatnonzero(got != ref)
            raise AssertionError(f"{label}: {f} differs at {bad.size} positions, first {bad[:5]}: "
                                 f"gpu {got[bad[:5]]} oracle {ref[bad[:5]]}")


def check(pol, p, label, flags=None, policy=0, priority=None, weights=None):
    say(f"[gpu] {label}: N={p.n_nodes} E={p.n_edges} W={p.n_workflows} M={p.n_instances} policy={policy}")
    if (policy & nalar.NALAR_ROUTE_WEIGHTED) and weights is None:
        weights = seeded_weights(p)
    assert_parity(gpu_run(pol, p, flags, policy, priority, weights),
                  oracle.run(p, policy=policy, priority=priority, weights=weights), label)


# ---------------------------------------------------------------- small cases

@pytest.mark.parametrize("name", golden_names())
def test_golden(policy, name):
    p, exp = load_golden(name)
    g = gpu_run(policy, p)
    assert g["status"] == exp["status"][0]
    assert g["rem"].tolist() == exp["rem"]
    assert g["order"].tolist() == exp["order"]
    assert g["slack"].tolist() == exp["slack"]
    assert g["route"].tolist() == exp["route"]
    assert g["cost"].tolist() == exp["cost"]


@pytest.mark.parametrize("seed", range(60))
def test_random_small_dags(policy, seed):
    rng = np.random.default_rng(1000 + seed)
    p = wl.random_dag(seed, n_nodes=int(rng.integers(1, 40)), n_workflows=int(rng.integers(1, 5)),
                      n_instances=int(rng.integers(0, 9)), n_types=int(rng.integers(1, 5)),
                      shuffle_ids=bool(seed % 2))
    check(policy, p, f"random_dag seed={seed}")


@pytest.mark.parametrize("seed", range(12))
def test_random_medium_dags(policy, policy_hbm, policy_hbm_levels, seed):
    """Several hundred futures per workflow, wide fan-in and fan-out (futures
    with more dependencies than a thread keeps in registers), ids shuffled
    (the HBM sweep then declines the ordered chunk pass) or in topological
    order (it takes it, with many rounds inside the one chunk)."""
    p = wl.random_dag(500 + seed, n_nodes=600, n_workflows=3, n_instances=40, n_types=6,
                      p_edge=0.02 + 0.01 * (seed % 4), est_max=10**9, load_max=10**12,
                      speed_hi=1 << 30, shuffle_ids=seed % 3 != 0)
    check(policy, p, f"medium seed={seed}")
    check(policy_hbm, p, f"medium seed={seed} hbm")
    check(policy_hbm_levels, p, f"medium seed={seed} hbm levels")


def chunked_workflows(seed, W=3, n=3000, heavy_every=60, p_near=0.3, p_done=0.3, sizes=None):
    """W workflows of n futures (or of the given sizes) with ids in
    topological order: each future
    depends on up to three earlier futures of its workflow, with probability
    p_near on one of the eight just before it (chains inside a chunk of
    positions), else anywhere earlier; about one in heavy_every depends on 40
    to 300 earlier ones (expanded by the whole workgroup).  Workflows above
    the LDS capacity take the HBM sweep without any flag."""
    rng = np.random.default_rng(seed)
    sizes = [n] * W if sizes is None else list(sizes)
    W = len(sizes)
    deps = []
    base = 0
    for w in range(W):
        n = sizes[w]
        if w:
            base += sizes[w - 1]
        for i in range(n):
            if i == 0:
                deps.append([])
            elif rng.random() < 1.0 / heavy_every and i >= 40:
                deps.append((base + rng.choice(i, size=int(rng.integers(40, min(300, i) + 1)),
                                               replace=False)).tolist())
            else:
                k = int(rng.integers(0, 4))
                near = rng.random(k) < p_near
                lo = np.maximum(0, i - 1 - rng.integers(0, 8, size=k))
                far = rng.integers(0, i, size=k)
                deps.append((base + np.where(near, lo, far)).tolist())
    N = sum(sizes)
    counts = np.array([len(d) for d in deps], np.int64)
    dep_off = np.zeros(N + 1, np.int32)
    dep_off[1:] = np.cumsum(counts)
    dep_idx = np.array([x for d in deps for x in d], np.int32)
    M, K = 24, 5
    return wl.Problem(f"chunked-{seed}", 1000, 150, np.repeat(np.arange(W), sizes).astype(np.int32),
                      rng.integers(0, K, size=N).astype(np.int32),
                      rng.integers(0, 10**6, size=N).astype(np.int64),
                      (rng.random(N) < p_done).astype(np.uint8),
                      np.where(rng.random(N) < 0.5, rng.integers(0, M, size=N), -1).astype(np.int32),
                      dep_off, dep_idx, (1000 + rng.integers(-10**5, 10**7, size=W)).astype(np.int64),
                      rng.integers(0, K, size=M).astype(np.int32),
                      rng.integers(0, 10**6, size=M).astype(np.int64),
                      rng.integers(500, 3000, size=M).astype(np.int32), wf_contiguous=True)


@pytest.mark.parametrize("seed", range(4))
def test_hbm_ordered_chunks(policy, policy_hbm, policy_hbm_levels, seed):
    """Workflows of 3,000 and 7,000 futures in topological id order: the
    ordered chunk pass (in-chunk chains, heavy futures inside a chunk, the
    last chunk ragged), against the level sweep and the LDS sweep; then the
    same with ids shuffled, where the ordered pass must decline."""
    p = chunked_workflows(seed, W=3, n=3000 if seed % 2 == 0 else 7000)
    check(policy, p, f"chunked seed={seed}")
    check(policy_hbm, p, f"chunked seed={seed} hbm")
    check(policy_hbm_levels, p, f"chunked seed={seed} hbm levels")
    q = wl.relabel(p, np.random.default_rng(seed).permutation(p.n_nodes))
    check(policy_hbm, q, f"chunked seed={seed} shuffled hbm")


def test_hbm_ordered_mixed_sizes(policy, policy_hbm_levels):
    """Small workflows beside one above the LDS capacity: one launch sweeps
    them all, the large one by the ordered pass with one future per thread
    per chunk."""
    for seed in range(3):
        p = chunked_workflows(20 + seed, sizes=[50, 700, 9000 + 37 * seed, 1200, 3])
        check(policy, p, f"mixed sizes seed={seed}")
        check(policy_hbm_levels, p, f"mixed sizes seed={seed} hbm levels")
        q = wl.relabel(p, np.random.default_rng(seed).permutation(p.n_nodes))
        check(policy, q, f"mixed sizes seed={seed} shuffled")


def test_hbm_ordered_many_heavy(policy_hbm, policy_hbm_levels):
    """More heavy futures in one chunk than the workgroup's list holds: the
    ones past it are pushed by their own threads."""
    p = chunked_workflows(11, W=2, n=2500, heavy_every=4)
    check(policy_hbm, p, "heavy chunks hbm")
    check(policy_hbm_levels, p, "heavy chunks hbm levels")


# ---------------------------------------------------------------- workloads

@pytest.mark.parametrize("name", ["tiny", "paper-scale", "deep-chains", "wide-mapreduce"])
def test_workloads(policy, name):
    check(policy, wl.WORKLOADS[name](), name)


@pytest.mark.parametrize("name", ["tiny", "paper-scale"])
def test_workloads_relabelled(policy, name):
    p = wl.WORKLOADS[name]()
    q = wl.relabel(p, np.random.default_rng(wl_index(name)).permutation(p.n_nodes))
    assert not q.wf_contiguous
    check(policy, q, f"{name} relabelled")


def test_contiguous_flag_not_set(policy):
    """The grouping path on ids that happen to be grouped already."""
    check(policy, wl.paper_scale(), "paper-scale grouped by the library", flags=0)


@pytest.mark.parametrize("name", ["tiny", "paper-scale", "wide-mapreduce"])
def test_workloads_hbm_sweep(policy_hbm, policy_hbm_levels, name):
    check(policy_hbm, wl.WORKLOADS[name](), f"{name} hbm")
    check(policy_hbm_levels, wl.WORKLOADS[name](), f"{name} hbm levels")


def test_deep_chains_hbm_small(policy_hbm, policy_hbm_levels):
    check(policy_hbm, wl.deep_chains(W=64), "deep chains W=64 hbm")
    check(policy_hbm_levels, wl.deep_chains(W=64), "deep chains W=64 hbm levels")


def test_deep_chains_hbm_full(policy_hbm):
    """The HBM sweep (state by position in global memory) on the full deep
    chains: 1,024 workflows of 128 levels each."""
    check(policy_hbm, wl.deep_chains(), "deep chains hbm")


@pytest.mark.parametrize("name", ["tiny", "paper-scale", "deep-chains"])
def test_workloads_tiled_sort(policy_tiled, name):
    check(policy_tiled, wl.WORKLOADS[name](), f"{name} tiled sort")


def test_workloads_relabelled_tiled_sort(policy_tiled):
    p = wl.tiny()
    check(policy_tiled, wl.relabel(p, np.random.default_rng(7).permutation(p.n_nodes)),
          "tiny relabelled tiled sort")


def _flat(deadline_offsets, per_wf=3):
    """Workflows of independent futures, none done, zero estimates: every
    future is ready and its slack is its workflow's deadline offset."""
    W = len(deadline_offsets)
    N = W * per_wf
    now = 1_000_000
    return wl.Problem("flat", now, 7, np.repeat(np.arange(W), per_wf).astype(np.int32),
                      np.zeros(N, np.int32), np.zeros(N, np.int64), np.zeros(N, np.uint8),
                      np.full(N, -1, np.int32), np.zeros(N + 1, np.int32), np.zeros(0, np.int32),
                      (now + np.asarray(deadline_offsets, np.int64)).astype(np.int64),
                      np.zeros(2, np.int32), np.array([5, 3], np.int64), np.array([1000, 7], np.int32),
                      wf_contiguous=True)


def test_sort_path_switching():
    """One handle through changing snapshots, so the host's choice between the
    bucketed sort (slack range guessed from the previous pass) and the tiled
    sort moves back and forth: first pass, overflowing buckets, a slack range
    far from the guess, more than 131072 ready futures, none ready."""
    p1 = wl.paper_scale()
    shifted = p1.copy(deadline_us=p1.deadline_us + 3_600_000_000)
    cases = [
        ("tiny first pass", wl.tiny()),
        ("tiny again", wl.tiny()),
        ("tiny other seed", wl.tiny(seed=3)),
        ("paper-scale after tiny", p1),
        ("paper-scale again", p1),
        ("paper-scale third", p1),
        ("all equal slack", _flat([3] * 200)),
        ("paper-scale", p1),
        ("deadlines shifted by an hour", shifted),
        ("shifted again", shifted),
        ("R=131072", wl.wide_mapreduce(W=32, fan=4096)),
        ("R=131072 again", wl.wide_mapreduce(W=32, fan=4096, seed=4)),
        ("R=262144", wl.wide_mapreduce(W=64, fan=4096)),
        ("paper-scale after R=262144", p1),
        ("none ready", p1.copy(done=np.ones(p1.n_nodes, np.uint8))),
        ("after none ready", p1),
        ("relabelled tiny", wl.relabel(wl.tiny(), np.random.default_rng(3).permutation(2048))),
        ("relabelled tiny again", wl.relabel(wl.tiny(), np.random.default_rng(4).permutation(2048))),
        ("range 2^40", _flat([-(1 << 39), 1 << 39, 0])),
        ("range 2^40 again", _flat([-(1 << 39), 1 << 39, 0])),
    ]
    with nalar.Policy() as pol:
        for label, p in cases:
            check(pol, p, label)


def test_large_ready_set_bins():
    """About a million ready futures on one handle: the first pass uses the
    tiled sort and leaves splitters, later passes the bin partition sort
    (the block sweep claims one segment per workflow and bin); every pass
    matches."""
    p = wl.wide_mapreduce()
    o = oracle.run(p)
    with nalar.Policy() as pol:
        pol.set_timing(True)
        for i in range(3):
            g = gpu_run(pol, p)
            assert_parity(g, o, f"wide map/reduce pass {i}")
            names = [n for n, _ in pol.timing()]
            say(f"[gpu] pass {i}: {names}")
            if i > 0:
                assert "sort_bin" in names and "sort_pass0" not in names


# ---------------------------------------------------------------- policy variants

VARIANTS = [nalar.NALAR_ORDER_LPT, nalar.NALAR_ROUTE_STATEFUL,
            nalar.NALAR_ORDER_LPT | nalar.NALAR_ROUTE_STATEFUL, nalar.NALAR_ROUTE_GREEDY,
            nalar.NALAR_ROUTE_GREEDY | nalar.NALAR_ROUTE_STATEFUL,
            nalar.NALAR_ROUTE_GREEDY | nalar.NALAR_ORDER_LPT,
            nalar.NALAR_ORDER_SRTF, nalar.NALAR_ORDER_SRTF | nalar.NALAR_ROUTE_STATEFUL,
            nalar.NALAR_ROUTE_WEIGHTED, nalar.NALAR_ROUTE_WEIGHTED | nalar.NALAR_ROUTE_STATEFUL,
            nalar.NALAR_ROUTE_WEIGHTED | nalar.NALAR_ORDER_SRTF]


@pytest.mark.parametrize("bits", VARIANTS)
@pytest.mark.parametrize("name", ["tiny", "paper-scale", "deep-chains", "wide-mapreduce"])
def test_policy_variants_workloads(policy, name, bits):
    p = wl.WORKLOADS[name]()
    check(policy, p, f"{name} policy {bits}", policy=bits)
    check(policy, p, f"{name} policy {bits} again", policy=bits)


@pytest.mark.parametrize("bits", VARIANTS)
def test_policy_variants_other_paths(policy_tiled, policy_hbm, bits):
    """Relabelled ids (grouping), the tiled sort, the HBM sweep and small
    random DAGs under each variant."""
    p = wl.tiny()
    q = wl.relabel(p, np.random.default_rng(9).permutation(p.n_nodes))
    check(policy_tiled, q, f"relabelled tiny tiled policy {bits}", policy=bits)
    check(policy_hbm, p, f"tiny hbm policy {bits}", policy=bits)
    for seed in range(8):
        d = wl.random_dag(700 + seed, n_nodes=120, n_workflows=3, n_instances=10, n_types=3,
                          shuffle_ids=bool(seed % 2))
        check(policy_tiled, d, f"random {seed} tiled policy {bits}", policy=bits)
        check(policy_hbm, d, f"random {seed} hbm policy {bits}", policy=bits)


def test_policy_switch_on_one_handle():
    """Changing the order key between passes on one handle: the bucket range
    planned from the previous pass's keys no longer fits, which the fallback
    must absorb."""
    p = wl.paper_scale()
    with nalar.Policy() as pol:
        for bits in (0, 0, nalar.NALAR_ORDER_LPT, nalar.NALAR_ORDER_LPT, 0, nalar.NALAR_ROUTE_STATEFUL):
            check(pol, p, f"switch policy {bits}", policy=bits)


@pytest.mark.parametrize("name", ["tiny", "paper-scale", "deep-chains", "wide-mapreduce"])
def test_priority_levels(policy, policy_tiled, policy_hbm, name):
    """Per-workflow priority levels (set_priority) with and without LPT, on
    every sort and sweep path, plus the level rule and keys near +-2^61."""
    p = wl.WORKLOADS[name]()
    rng = np.random.default_rng(20 + wl_index(name))
    for levels in (rng.integers(0, 16, p.n_workflows), rng.integers(0, 2, p.n_workflows),
                   np.full(p.n_workflows, 15)):
        pr = levels.astype(np.uint8)
        check(policy, p, f"{name} levels", priority=pr)
        check(policy, p, f"{name} levels lpt", policy=nalar.NALAR_ORDER_LPT, priority=pr)
    if name == "tiny":
        pr = rng.integers(0, 16, p.n_workflows).astype(np.uint8)
        q = wl.relabel(p, np.random.default_rng(5).permutation(p.n_nodes))
        check(policy_tiled, q, "relabelled levels", priority=pr)
        check(policy_hbm, p, "hbm levels", priority=pr)
        bad = pr.copy()
        bad[7] = 16
        check(policy, p, "level 16", priority=bad)
        # slacks near -2^61 - rem and +2^61: the order by (-level, key, wf, id)
        # needs no bound on the key
        dl = p.now_us + rng.choice([-(1 << 61), (1 << 61) - (1 << 40), 0, 1 << 58], p.n_workflows)
        far = p.copy(deadline_us=dl.astype(np.int64))
        for pol, name in ((policy, "default"), (policy_tiled, "tiled"), (policy_hbm, "hbm")):
            for bits in (0, nalar.NALAR_ORDER_SRTF):
                check(pol, far, f"keys near 2^61 with levels {name} {bits}", policy=bits, priority=pr)
                check(pol, far, f"keys near 2^61 with levels {name} {bits} again", policy=bits, priority=pr)
            check(pol, far, f"keys near 2^61 without levels {name}")


def test_priority_levels_bucketed():
    """Repeated passes with priority levels on one handle: after the first pass
    the bucketed sort maps each level to its own group of buckets.  Level sets
    then move above and below the planned groups (keys clamped to the end
    buckets, a few of them or whole levels that overflow and fall back), with
    and without LPT; every pass must match the oracle."""
    p = wl.paper_scale()
    rng = np.random.default_rng(77)
    base = rng.integers(2, 6, p.n_workflows).astype(np.uint8)
    mixed = base.copy()
    mixed[[3, 500, 2000]] = 0
    mixed[[7, 1000]] = 1
    mixed[[11, 3000, 4095]] = 12
    seq = [(base, 0), (base, 0), (base, 0), (mixed, 0), (base + 6, 0), (base, 0),
           (base, nalar.NALAR_ORDER_LPT), (base, nalar.NALAR_ORDER_LPT), (mixed, nalar.NALAR_ORDER_LPT)]
    with nalar.Policy() as pol:
        pol.set_timing(True)
        bucketed = 0
        for i, (pr, bits) in enumerate(seq):
            check(pol, p, f"levels pass {i} policy {bits}", policy=bits, priority=pr)
            names = [n for n, _ in pol.timing()]
            if "sort_bucket" in names and "sort_pass0" not in names:
                bucketed += 1
        assert bucketed >= 3, f"only {bucketed} level passes took the bucketed sort"


def test_lpt_repeated_bucketed():
    """LPT's long-tailed key at paper scale on one handle: the first passes
    overflow the base plan and settle on denser buckets (the large-bucket
    kernels, whose busiest group holds more futures than one LDS chunk);
    every pass must match the oracle and most must take the bucketed sort."""
    p = wl.paper_scale()
    with nalar.Policy() as pol:
        pol.set_timing(True)
        bucketed = 0
        for i in range(8):
            check(pol, p, f"lpt pass {i}", policy=nalar.NALAR_ORDER_LPT)
            names = [n for n, _ in pol.timing()]
            if "sort_bucket" in names and "sort_pass0" not in names:
                bucketed += 1
        assert bucketed >= 5, f"only {bucketed} LPT passes took the bucketed sort"


def test_policy_unknown_bits_rejected(policy):
    dp = nalar.DeviceProblem.from_host(wl.tiny())
    out = nalar.DeviceResult.alloc(dp.n_nodes)
    assert policy.run_pass(dp, out, policy=64) == nalar.NALAR_EINVAL
    assert policy.run_pass(dp, out, policy=nalar.NALAR_ORDER_LPT | nalar.NALAR_ORDER_SRTF) == nalar.NALAR_EINVAL
    assert policy.run_pass(dp, out, policy=nalar.NALAR_ROUTE_WEIGHTED) == nalar.NALAR_EINVAL  # no weights


def test_weighted_rules_and_precedence(policy, policy_tiled):
    """Weights above NALAR_WEIGHT_MAX and weighted with greedy routing are
    EINVAL, and a bad weight wins over a cycle (EINVAL before ECYCLE); all-zero
    weights give the default routes; repeated weighted passes on one handle
    (the bucketed sort after the first) match the oracle."""
    p = wl.tiny()
    W = nalar.NALAR_ROUTE_WEIGHTED
    big = seeded_weights(p)
    big[3] = (1 << 20) + 1
    check(policy, p, "weight above max", policy=W, weights=big)
    check(policy_tiled, p, "weight above max tiled", policy=W, weights=big)
    check(policy, p, "weighted with greedy", policy=W | nalar.NALAR_ROUTE_GREEDY, weights=seeded_weights(p))
    cyc = p.copy(dep_idx=p.dep_idx.copy())
    v = int(np.flatnonzero(np.diff(p.dep_off) > 0)[0])
    cyc.dep_idx[p.dep_off[v]] = v  # a self-dependency
    check(policy, cyc, "cycle without weights")
    check(policy, cyc, "cycle and bad weight", policy=W, weights=big)
    check(policy, p, "zero weights", policy=W, weights=np.zeros(p.n_instances, np.uint32))
    q = wl.paper_scale()
    for i in range(4):
        check(policy, q, f"weighted paper scale pass {i}", policy=W)
    r = wl.relabel(p, np.random.default_rng(3).permutation(p.n_nodes))
    check(policy_tiled, r, "weighted relabelled tiled", policy=W | nalar.NALAR_ROUTE_STATEFUL)


@pytest.mark.parametrize("m,n_types", [(1, 1), (63, 2), (1024, 1), (1024, 300)])
def test_weighted_instance_tables(policy, m, n_types):
    """Weighted routing with one instance, many types, and the largest tables
    (one type of 1024 instances, 300 types), weights up to the maximum."""
    p = wl.windowed(64)
    rng = np.random.default_rng(m + n_types)
    q = p.copy(inst_type=rng.integers(0, n_types, m).astype(np.int32),
               inst_load_us=rng.integers(0, 2_000_000, m).astype(np.int64),
               inst_speed_permille=rng.integers(500, 2001, m).astype(np.int32),
               type=rng.integers(0, n_types + 1, p.n_nodes).astype(np.int32),
               loc=np.where(rng.random(p.n_nodes) < 0.5, rng.integers(0, m, p.n_nodes), -1).astype(np.int32))
    w = rng.choice([0, 1, 7, 1 << 20], m).astype(np.uint32)
    check(policy, q, f"weighted M={m} types={n_types}", policy=nalar.NALAR_ROUTE_WEIGHTED, weights=w)


def _one_type(n_inst, loads, speeds, est, loc=None, mig=200_000):
    N = len(est)
    now = 1_000
    dl = 1_000_000 + np.random.default_rng(N).permutation(N).astype(np.int64) * 1000
    return wl.Problem("one-type", now, mig, np.arange(N, dtype=np.int32), np.zeros(N, np.int32),
                      np.asarray(est, np.int64), np.zeros(N, np.uint8),
                      np.full(N, -1, np.int32) if loc is None else np.asarray(loc, np.int32),
                      np.zeros(N + 1, np.int32), np.zeros(0, np.int32), (now + dl).astype(np.int64),
                      np.zeros(n_inst, np.int32), np.asarray(loads, np.int64),
                      np.asarray(speeds, np.int32), wf_contiguous=True)


def test_greedy_many_candidates_and_overflow(policy):
    """More candidates of one type than lanes in a wave (the candidate loop),
    identical instances (every decision a tie), and a load overflow (ERANGE)."""
    rng = np.random.default_rng(4)
    G = nalar.NALAR_ROUTE_GREEDY
    p = _one_type(300, rng.integers(0, 10**6, 300), rng.integers(500, 2000, 300),
                  rng.integers(0, 10**6, 2000), loc=np.where(rng.random(2000) < 0.5, rng.integers(0, 300, 2000), -1))
    check(policy, p, "greedy 300 candidates", policy=G)
    check(policy, p, "greedy 300 candidates stateful", policy=G | nalar.NALAR_ROUTE_STATEFUL)
    q = _one_type(5, [700] * 5, [1000] * 5, [33] * 500)
    check(policy, q, "greedy identical instances", policy=G)
    o = _one_type(1, [1 << 60], [1], [1 << 40] * 3200)
    check(policy, o, "greedy load overflow", policy=G)
    check(policy, wl.tiny(), "after greedy overflow")


@pytest.mark.parametrize("n_inst", [1, 7, 8, 9, 16, 17, 63, 64, 65])
def test_greedy_candidate_counts(policy, n_inst):
    """Load-aware routing around every width the kernel distinguishes (up to
    8, 16 and 64 candidates in registers, more in LDS), with enough futures of
    the type to wrap its queue and leave a partial last batch; plain, pinned
    (stateful) and with heavy ties (equal speeds and loads)."""
    rng = np.random.default_rng(40 + n_inst)
    G = nalar.NALAR_ROUTE_GREEDY
    n = 777
    loc = np.where(rng.random(n) < 0.4, rng.integers(0, n_inst, n), -1)
    p = _one_type(n_inst, rng.integers(0, 10**6, n_inst), rng.integers(300, 3000, n_inst),
                  rng.integers(0, 10**5, n), loc=loc)
    check(policy, p, f"greedy {n_inst} candidates", policy=G)
    check(policy, p, f"greedy {n_inst} candidates stateful", policy=G | nalar.NALAR_ROUTE_STATEFUL)
    q = _one_type(n_inst, [500] * n_inst, [1000] * n_inst, rng.integers(1, 4, n) * 10, loc=loc)
    check(policy, q, f"greedy {n_inst} tied candidates", policy=G)


def _sized_workflows(sizes, seed, heavy_every=7):
    """Contiguous workflows of the given sizes; every future depends on up to
    three earlier futures of its workflow, every heavy_every-th on up to six."""
    rng = np.random.default_rng(seed)
    W = len(sizes)
    wf = np.repeat(np.arange(W, dtype=np.int32), sizes)
    starts = np.concatenate([[0], np.cumsum(sizes)])
    counts, flat = [], []
    for w in range(W):
        for i in range(sizes[w]):
            cap = 6 if i % heavy_every == heavy_every - 1 else 3
            k = int(rng.integers(0, min(i, cap) + 1))
            par = rng.choice(i, size=k, replace=False) if k else []
            counts.append(k)
            flat.extend(int(starts[w] + q) for q in par)
    N = int(starts[-1])
    dep_off = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    M, K = 16, 4
    now = 5_000
    return wl.Problem("sized", now, 150_000, wf, rng.integers(0, K, N).astype(np.int32),
                      rng.integers(0, 10**5, N).astype(np.int64), (rng.random(N) < 0.3).astype(np.uint8),
                      np.where(rng.random(N) < 0.5, rng.integers(0, M, N), -1).astype(np.int32),
                      dep_off, np.asarray(flat, np.int32),
                      (now + rng.integers(-10**5, 10**7, W)).astype(np.int64),
                      (np.arange(M) % K).astype(np.int32), rng.integers(0, 10**6, M).astype(np.int64),
                      rng.integers(200, 3000, M).astype(np.int32), wf_contiguous=True)


def test_grouped_waves(policy, policy_tiled, policy_hbm):
    """Workflows of at most 32 futures on average are swept two per wave:
    pairs that fill a slice exactly, pairs too large for one slice (swept one
    by one), empty workflows, an odd count (a last group of one), relabelled
    ids, every policy variant and levels; and a dependency on the other
    workflow of a pair (light and heavy futures) is an error."""
    sizes = [30, 34, 64, 1, 0, 63, 2, 33, 31, 5, 27, 3, 29, 20, 12, 32, 32]
    p = _sized_workflows(sizes, 3)
    check(policy, p, "grouped sizes")
    check(policy_tiled, p, "grouped sizes tiled")
    check(policy_hbm, p, "grouped sizes hbm")
    q = wl.relabel(p, np.random.default_rng(2).permutation(p.n_nodes))
    check(policy, q, "grouped sizes relabelled")
    for bits in VARIANTS:
        check(policy, p, f"grouped sizes policy {bits}", policy=bits)
    lv = np.random.default_rng(4).integers(0, 5, len(sizes)).astype(np.uint8)
    check(policy, p, "grouped sizes levels", priority=lv)
    starts = np.concatenate([[0], np.cumsum(sizes)])
    for label, w_from, w_to in (("wf1 -> wf0", 1, 0), ("wf0 -> wf1", 0, 1), ("wf8 -> wf7", 8, 7)):
        bad = p.copy(dep_idx=p.dep_idx.copy())
        v = int(starts[w_from]) + 10           # a future with dependencies
        assert bad.dep_off[v + 1] > bad.dep_off[v], label
        bad.dep_idx[bad.dep_off[v]] = int(starts[w_to]) + 1
        check(policy, bad, f"cross-workflow dependency {label}")
    hv = next(v for v in range(int(starts[1]), int(starts[2])) if p.dep_off[v + 1] - p.dep_off[v] > 3)
    bad = p.copy(dep_idx=p.dep_idx.copy())
    bad.dep_idx[bad.dep_off[hv + 1] - 1] = 2
    check(policy, bad, "cross-workflow dependency of a heavy future")


@pytest.mark.parametrize("seed", range(12))
def test_grouped_waves_random_sizes(policy, seed):
    """Random workflow sizes around the pair boundary (a pair fills one
    64-future slice, or spills and is swept one workflow at a time), averaging
    at most 32 futures, with random levels and policy variants."""
    rng = np.random.default_rng(500 + seed)
    W = int(rng.integers(2, 90))
    sizes = [int(x) for x in rng.choice([0, 1, 5, 16, 31, 32, 33, 40, 63, 64], size=W,
                                        p=[.05, .05, .1, .15, .15, .2, .1, .1, .05, .05])]
    while sum(sizes) > 32 * W:  # keep the pairs' plan (average at most 32)
        sizes[int(np.argmax(sizes))] //= 2
    p = _sized_workflows(sizes, 600 + seed, heavy_every=int(rng.integers(3, 9)))
    bits = [0, nalar.NALAR_ORDER_LPT, nalar.NALAR_ROUTE_STATEFUL][seed % 3]
    check(policy, p, f"random sizes seed {seed}", policy=bits)
    lv = rng.integers(0, 4, W).astype(np.uint8)
    check(policy, p, f"random sizes seed {seed} levels", policy=bits, priority=lv)


@pytest.mark.parametrize("seed", range(6))
def test_frontier_rounds(policy, policy_tiled, seed):
    """Workflows of 70-512 futures (four or eight futures per lane, whose
    rounds follow a frontier), with futures of up to six dependencies pushed
    by the whole wave, duplicate-free random DAGs, and cycle / cross-workflow
    errors planted in them."""
    rng = np.random.default_rng(900 + seed)
    W = int(rng.integers(3, 40))
    lo, hi = ((70, 180), (257, 512), (130, 512))[seed % 3]
    sizes = [int(x) for x in rng.integers(lo, hi + 1, W)]
    p = _sized_workflows(sizes, 1000 + seed, heavy_every=int(rng.integers(2, 6)))
    check(policy, p, f"frontier seed {seed}")
    check(policy_tiled, p, f"frontier seed {seed} tiled", policy=nalar.NALAR_ORDER_LPT)
    starts = np.concatenate([[0], np.cumsum(sizes)])
    v = int(starts[1]) + 5  # a cycle: future v depends on a later future of its workflow that depends on v
    later = int(starts[1]) + 100
    bad = p.copy(dep_idx=p.dep_idx.copy())
    if bad.dep_off[v + 1] > bad.dep_off[v] and bad.dep_off[later + 1] > bad.dep_off[later]:
        bad.dep_idx[bad.dep_off[v]] = later
        bad.dep_idx[bad.dep_off[later]] = v
        check(policy, bad, f"frontier seed {seed} cycle")


def test_other_seeds(policy):
    for s in (11, 12):
        check(policy, wl.paper_scale(seed=s), f"paper-scale seed {s}")
        check(policy, wl.wide_mapreduce(seed=s, W=32, fan=1000), f"mapreduce seed {s}")


def test_repeat_is_deterministic(policy):
    p = wl.wide_mapreduce(W=64)
    a = gpu_run(policy, p)
    for _ in range(3):
        b = gpu_run(policy, p)
        for f in ("rem", "order", "slack", "route", "cost"):
            assert np.array_equal(a[f], b[f])


def test_scratch_reuse_across_sizes(policy):
    for p in (wl.tiny(), wl.wide_mapreduce(W=64), wl.tiny(seed=3), wl.paper_scale(),
              wl.random_dag(5, n_nodes=30, n_workflows=2)):
        check(policy, p, f"reuse {p.name}")


def test_fresh_handle_each_call():
    for _ in range(3):
        with nalar.Policy() as pol:
            check(pol, wl.tiny(), "fresh handle")


# ---------------------------------------------------------------- degenerate

def test_degenerate_cases(policy):
    base = wl.tiny()
    N = base.n_nodes
    cases = {
        "all done": base.copy(done=np.ones(N, np.uint8)),
        "no edges": base.copy(dep_off=np.zeros(N + 1, np.int32), dep_idx=np.zeros(0, np.int32),
                              done=np.zeros(N, np.uint8)),
        "no instances": base.copy(inst_type=np.zeros(0, np.int32), inst_load_us=np.zeros(0, np.int64),
                                  inst_speed_permille=np.zeros(0, np.int32),
                                  loc=np.full(N, -1, np.int32)),
        "one instance": base.copy(inst_type=np.zeros(1, np.int32), inst_load_us=np.zeros(1, np.int64),
                                  inst_speed_permille=np.ones(1, np.int32),
                                  loc=np.where(base.loc >= 0, 0, -1).astype(np.int32)),
        "equal slack": base.copy(est_us=np.ones(N, np.int64), deadline_us=np.full(64, base.now_us + 10**6)),
        "zero est": base.copy(est_us=np.zeros(N, np.int64)),
        "negative slack": base.copy(deadline_us=base.deadline_us - 10**9),
        "max est": base.copy(est_us=np.full(N, 1 << 40, np.int64)),
        "max load": base.copy(inst_load_us=np.full(base.n_instances, 1 << 60, np.int64),
                              migration_cost_us=1 << 60),
        "single workflow": base.copy(wf=np.zeros(N, np.int32), deadline_us=base.deadline_us[:1].copy(),
                                     dep_off=np.zeros(N + 1, np.int32), dep_idx=np.zeros(0, np.int32)),
    }
    for label, p in cases.items():
        check(policy, p, label)


def test_empty_and_single(policy):
    one = wl.Problem("one", 10, 7, np.zeros(1, np.int32), np.zeros(1, np.int32),
                     np.array([5], np.int64), np.zeros(1, np.uint8), np.array([0], np.int32),
                     np.array([0, 0], np.int32), np.zeros(0, np.int32), np.array([20], np.int64),
                     np.array([0], np.int32), np.array([3], np.int64), np.array([1000], np.int32), True)
    check(policy, one, "single future")
    empty = one.copy(wf=np.zeros(0, np.int32), type=np.zeros(0, np.int32), est_us=np.zeros(0, np.int64),
                     done=np.zeros(0, np.uint8), loc=np.zeros(0, np.int32), dep_off=np.array([0], np.int32))
    check(policy, empty, "no futures")
    nowf = empty.copy(deadline_us=np.zeros(0, np.int64))
    check(policy, nowf, "no futures, no workflows")


# ---------------------------------------------------------------- errors

ERROR_CASES = [
    ("wf", 5, -1), ("wf", 5, 64), ("type", 3, -1), ("loc", 7, -2), ("loc", 7, 16),
    ("est_us", 9, -1), ("est_us", 9, (1 << 40) + 1), ("done", 4, 2),
    ("dep_idx", 10, -1), ("dep_idx", 10, 2048), ("dep_idx", 10, 40),
    ("dep_off", 0, 1), ("dep_off", 2048, 1), ("inst_type", 0, -1),
    ("inst_speed_permille", 2, 0), ("inst_load_us", 1, -1), ("inst_load_us", 1, (1 << 60) + 1),
    ("deadline_us", 3, wl.NOW_US + (1 << 61) + 1),
]


@pytest.mark.parametrize("case", ERROR_CASES)
def test_error_rules(policy, case):
    field, idx, value = case
    p = wl.tiny().copy()
    getattr(p, field)[idx] = value
    check(policy, p, f"error {case}")
    q = wl.relabel(wl.tiny(), np.random.default_rng(9).permutation(2048)).copy()
    if field in ("dep_off", "dep_idx"):
        return
    getattr(q, field)[idx] = value
    check(policy, q, f"error {case} relabelled")


@pytest.mark.parametrize("case", ERROR_CASES)
def test_error_rules_hbm_sweep(policy_hbm, case):
    """The same rules when every workflow takes the workgroup (HBM) path."""
    field, idx, value = case
    p = wl.tiny().copy()
    getattr(p, field)[idx] = value
    check(policy_hbm, p, f"error {case} hbm")


def _mixed_sizes(sizes, seed, n_instances=24, n_types=5):
    """Workflows of the given sizes, ids grouped by workflow; future i of a
    workflow depends on up to three of the four futures before it."""
    rng = np.random.default_rng(seed)
    W = len(sizes)
    N = int(sum(sizes))
    wf = np.repeat(np.arange(W), sizes).astype(np.int32)
    starts = np.r_[0, np.cumsum(sizes)[:-1]]
    deps, off = [], [0]
    for w, n in enumerate(sizes):
        for i in range(n):
            k = int(rng.integers(0, min(i, 3) + 1))
            par = rng.choice(np.arange(max(0, i - 4), i), size=k, replace=False) if k else []
            deps.extend(int(starts[w] + q) for q in sorted(par))
            off.append(len(deps))
    types = rng.integers(0, n_types, N).astype(np.int32)
    est = rng.integers(1, 10**6, N).astype(np.int64)
    done = (rng.random(N) < 0.2).astype(np.uint8)
    loc = np.where(rng.random(N) < 0.5, rng.integers(0, n_instances, N), -1).astype(np.int32)
    now = 10**12
    return wl.Problem("mixed", now, 5000, wf, types, est, done, loc, np.array(off, np.int32),
                      np.array(deps, np.int32), now + rng.integers(10**6, 10**8, W).astype(np.int64),
                      rng.integers(0, n_types, n_instances).astype(np.int32),
                      rng.integers(0, 10**6, n_instances).astype(np.int64),
                      rng.integers(1, 3000, n_instances).astype(np.int32), wf_contiguous=True)


def test_mixed_workflow_sizes(policy):
    """Small workflows with a few far larger than a wave's slice: the large
    ones are swept by whole workgroups in the same launch."""
    sizes = [8] * 300 + [2000] + [8] * 100 + [700, 3] + [1] * 50
    p = _mixed_sizes(sizes, 1)
    check(policy, p, "mixed sizes")
    for field, idx, value in (("type", 300 * 8 + 1500, -1), ("loc", 300 * 8 + 10, 24),
                              ("est_us", 300 * 8 + 2000 + 8 * 100 + 650, -5),
                              ("done", 5, 3), ("wf", 300 * 8 + 1999, 302),
                              ("deadline_us", 300, 1 << 62)):
        q = p.copy()
        getattr(q, field)[idx] = value
        check(policy, q, f"mixed sizes, {field}[{idx}] = {value}")


def test_error_cycle_and_self_loop(policy, policy_hbm):
    p = wl.tiny().copy()
    p.dep_idx[p.dep_off[12]] = 12
    check(policy, p, "self loop")
    check(policy_hbm, p, "self loop hbm")
    c = wl.Problem("cyc", 0, 0, np.zeros(3, np.int32), np.zeros(3, np.int32), np.ones(3, np.int64),
                   np.zeros(3, np.uint8), -np.ones(3, np.int32), np.array([0, 1, 2, 3], np.int32),
                   np.array([2, 0, 1], np.int32), np.array([100], np.int64), np.zeros(0, np.int32),
                   np.zeros(0, np.int64), np.zeros(0, np.int32), True)
    check(policy, c, "3-cycle")
    check(policy_hbm, c, "3-cycle hbm")


def test_error_contiguous_promise_broken(policy):
    p = wl.relabel(wl.tiny(), np.random.default_rng(2).permutation(2048))
    g = gpu_run(policy, p, flags=nalar.NALAR_WF_CONTIGUOUS)
    assert g["status"] == nalar.NALAR_EINVAL


def test_error_overflow_and_precedence(policy):
    n = (1 << 22) + 1
    chain = wl.Problem("chain", 0, 0, np.zeros(n, np.int32), np.zeros(n, np.int32),
                       np.full(n, 1 << 40, np.int64), np.zeros(n, np.uint8), -np.ones(n, np.int32),
                       np.r_[0, 0, np.arange(1, n)].astype(np.int32), np.arange(n - 1).astype(np.int32),
                       np.array([0], np.int64), np.zeros(0, np.int32), np.zeros(0, np.int64),
                       np.zeros(0, np.int32), True)
    check(policy, chain, "overflowing chain")
    cyc = chain.copy()
    cyc.dep_idx[0] = 5
    check(policy, cyc, "cycle beats overflow")


def test_handle_usable_after_error(policy):
    p = wl.tiny().copy()
    p.type[0] = -1
    assert gpu_run(policy, p)["status"] == nalar.NALAR_EINVAL
    check(policy, wl.tiny(), "after error")


def test_null_arguments(policy):
    dp = nalar.DeviceProblem.from_host(wl.tiny())
    out = nalar.DeviceResult.alloc(dp.n_nodes)
    raw = dp.c_struct()
    raw.dep_idx = None
    assert policy.run_pass(dp, out, raw=raw) == nalar.NALAR_EINVAL
    raw = dp.c_struct()
    raw.reserved = 1
    assert policy.run_pass(dp, out, raw=raw) == nalar.NALAR_EINVAL
    cr = out.c_struct()
    cr.order = None
    assert nalar.nalar_policy_pass(policy.handle, dp.c_struct(), cr) == nalar.NALAR_EINVAL


# ---------------------------------------------------------------- dynamic stream

_stream_state = {}


def _stream():
    if "it" not in _stream_state:
        _stream_state["it"] = wl.dynamic_stream(steps=100)
        _stream_state["next"] = 0
    return _stream_state


@pytest.mark.parametrize("chunk", range(11))
def test_dynamic_stream_every_step(policy, chunk):
    """Steps 0..100 of the evolving map/reduce graph, bit-exact at every step."""
    st = _stream()
    lo, hi = chunk * 10, min(chunk * 10 + 9, 100) if chunk < 10 else 100
    if chunk == 10:
        lo = 100
    assert st["next"] == lo, "dynamic stream chunks must run in order"
    pool = cf.ThreadPoolExecutor(max_workers=8)
    futs = []
    for step in range(lo, hi + 1):
        snap = next(st["it"]).copy()
        st["next"] = step + 1
        say(f"[gpu] dynamic step {step}: N={snap.n_nodes}")
        g = gpu_run(policy, snap)
        futs.append((step, g, pool.submit(oracle.run, snap)))
    for step, g, f in futs:
        assert_parity(g, f.result(), f"dynamic step {step}")
    pool.shutdown()


# ---------------------------------------------------------------- graph store

def _store_step(st, p, prev_n, prev_done):
    """Feed snapshot p to the store as the delta from the previous one."""
    N = p.n_nodes
    if prev_n == 0:
        assert st.set_workflows(p.deadline_us) == nalar.NALAR_OK
        assert st.set_instances(p.inst_type, p.inst_load_us, p.inst_speed_permille) == nalar.NALAR_OK
    else:
        newly = np.flatnonzero((p.done[:prev_n] == 1) & (prev_done == 0)).astype(np.int32)
        assert st.complete(newly) == nalar.NALAR_OK
    e0, e1 = int(p.dep_off[prev_n]), int(p.dep_off[N])
    rc = st.append(p.wf[prev_n:N], p.type[prev_n:N], p.est_us[prev_n:N], p.done[prev_n:N],
                   p.loc[prev_n:N], p.dep_off[prev_n:N + 1] - e0, p.dep_idx[e0:e1],
                   contiguous=bool(p.wf_contiguous))
    assert rc == nalar.NALAR_OK
    return N, p.done[:N].copy()


def test_store_follows_dynamic_stream():
    """The evolving map/reduce graph fed to the device-resident store as
    deltas (completions, appended futures): every pass over the store equals
    the oracle on the full snapshot."""
    with nalar.Policy() as pol:
        st = nalar.Store(pol)
        try:
            prev_n, prev_done = 0, None
            for step, p in enumerate(wl.dynamic_stream(steps=30)):
                prev_n, prev_done = _store_step(st, p, prev_n, prev_done)
                assert st.n_nodes == p.n_nodes
                if step % 3 == 0 or step == 30:
                    out = nalar.DeviceResult.alloc(p.n_nodes)
                    rc = st.run_pass(out, p.now_us, p.migration_cost_us)
                    torch.cuda.synchronize()
                    R = out.n_ready
                    g = dict(status=rc, n_ready=R, rem=out.rem[:p.n_nodes].cpu().numpy(),
                             order=out.order[:R].cpu().numpy(), slack=out.slack[:R].cpu().numpy(),
                             route=out.route[:R].cpu().numpy(), cost=out.cost[:R].cpu().numpy(),
                             err=pol.last_error())
                    say(f"[gpu] store step {step}: N={p.n_nodes}")
                    assert_parity(g, oracle.run(p), f"store step {step}")
        finally:
            st.close()


def test_store_small_graphs_and_errors():
    """Random DAGs built up in several appends (ids contiguous or not, policy
    variants), an out-of-range completion reported by the next pass only, and
    argument errors."""
    with nalar.Policy() as pol:
        for seed in range(6):
            p = wl.random_dag(900 + seed, n_nodes=200, n_workflows=4, n_instances=12, n_types=3,
                              shuffle_ids=bool(seed % 2))
            st = nalar.Store(pol)
            try:
                assert st.set_workflows(p.deadline_us) == 0
                assert st.set_instances(p.inst_type, p.inst_load_us, p.inst_speed_permille) == 0
                cuts = [0, 37, 120, 120, 200]
                for a, b in zip(cuts, cuts[1:]):
                    e0, e1 = int(p.dep_off[a]), int(p.dep_off[b])
                    assert st.append(p.wf[a:b], p.type[a:b], p.est_us[a:b], p.done[a:b], p.loc[a:b],
                                     p.dep_off[a:b + 1] - e0, p.dep_idx[e0:e1],
                                     contiguous=bool(p.wf_contiguous)) == 0
                for bits in (0, nalar.NALAR_ORDER_LPT | nalar.NALAR_ROUTE_GREEDY):
                    out = nalar.DeviceResult.alloc(p.n_nodes)
                    rc = st.run_pass(out, p.now_us, p.migration_cost_us, policy=bits)
                    torch.cuda.synchronize()
                    R = out.n_ready
                    g = dict(status=rc, n_ready=R, rem=out.rem[:p.n_nodes].cpu().numpy(),
                             order=out.order[:R].cpu().numpy(), slack=out.slack[:R].cpu().numpy(),
                             route=out.route[:R].cpu().numpy(), cost=out.cost[:R].cpu().numpy(),
                             err=pol.last_error())
                    assert_parity(g, oracle.run(p, policy=bits), f"store seed {seed} policy {bits}")
                # an id out of range: the next pass fails, the one after is fine
                assert st.complete(np.array([p.n_nodes + 5], np.int32)) == 0
                out = nalar.DeviceResult.alloc(p.n_nodes)
                assert st.run_pass(out, p.now_us, p.migration_cost_us) == nalar.NALAR_EINVAL
                rc = st.run_pass(out, p.now_us, p.migration_cost_us)
                assert rc == nalar.NALAR_OK, pol.last_error()
                # argument errors
                z = np.zeros(0, np.int32)
                assert nalar.nalar_store_append(st.handle, -1, 0, None, None, None, None, None, None,
                                                None, 0) == nalar.NALAR_EINVAL
                assert nalar.nalar_store_append(st.handle, 1, 0, None, None, None, None, None, None,
                                                None, 0) == nalar.NALAR_EINVAL
                assert nalar.nalar_store_complete(st.handle, -1, None) == nalar.NALAR_EINVAL
                assert nalar.nalar_store_pass(st.handle, 0, 0, 64, out.c_struct()) == nalar.NALAR_EINVAL
                assert nalar.nalar_store_pass(st.handle, 0, 0, nalar.NALAR_ROUTE_WEIGHTED,
                                              out.c_struct()) == nalar.NALAR_EINVAL
                del z
            finally:
                st.close()


# ------------------------------------------------------- large instance tables

@pytest.mark.parametrize("n_inst,n_types", [(255, 3), (257, 70), (1021, 200), (1024, 5), (1024, 1)])
@pytest.mark.parametrize("shuffle", [False, True])
def test_large_instance_tables(policy, n_inst, n_types, shuffle):
    """Instance tables past one workgroup's threads and past the directly
    indexed types, sizes not a multiple of four: the (type, index) ranking and
    the per-type runs, under plain, stateful and greedy routing."""
    p = wl.random_dag(900 + n_inst + n_types, n_nodes=500, n_workflows=3, n_instances=n_inst,
                      n_types=n_types, p_edge=0.02, est_max=10**6, load_max=10**9,
                      shuffle_ids=shuffle)
    for pol_bits in (0, nalar.NALAR_ROUTE_STATEFUL, nalar.NALAR_ROUTE_GREEDY):
        check(policy, p, f"instances={n_inst} types={n_types} shuffle={shuffle}", policy=pol_bits)


# ------------------------------------------------------------ bin partition sort

def _independent(W, n, seed, spread=True):
    """W workflows of n independent futures (no dependencies, none done): all
    ready, keys from seeded service times and deadlines."""
    rng = np.random.default_rng(seed)
    N = W * n
    p = wl.random_dag(seed, n_nodes=4, n_workflows=1, n_instances=24, n_types=5)
    types = rng.integers(0, 6, N).astype(np.int32)
    M = p.n_instances
    return wl.Problem(f"independent-{W}x{n}", p.now_us, 200_000, np.repeat(np.arange(W), n).astype(np.int32),
                      types, rng.integers(1, 10**7, N).astype(np.int64), np.zeros(N, np.uint8),
                      np.where(rng.random(N) < 0.5, rng.integers(0, M, N), -1).astype(np.int32),
                      np.zeros(N + 1, np.int32), np.zeros(0, np.int32),
                      (p.now_us + (rng.integers(2_000_000, 20_000_000, W) if spread else
                                   np.full(W, 5_000_000))).astype(np.int64),
                      rng.integers(0, 5, M).astype(np.int32), rng.integers(0, 2_000_000, M).astype(np.int64),
                      rng.integers(500, 2001, M).astype(np.int32), wf_contiguous=True)


def _sort_kind(pol):
    names = [n for n, _ in pol.timing()]
    return "bin" if "sort_bin" in names else ("bucket" if "sort_bucket" in names and "sort_pass0" not in names
                                                else "tiled")


def test_bin_sort_wide_mapreduce():
    """Repeated passes over the wide map/reduce snapshot on one handle: the
    first pass takes the tiled sort and leaves splitters, the later ones the
    bin partition sort; then a policy switch (other keys, overflowing bins,
    fallback) and back."""
    p = wl.wide_mapreduce()
    ref = {b: oracle.run(p, policy=b) for b in (0, nalar.NALAR_ORDER_SRTF, nalar.NALAR_ORDER_LPT)}
    kinds = []
    with nalar.Policy() as pol:
        pol.set_timing(True)
        for i, bits in enumerate([0, 0, 0, nalar.NALAR_ORDER_SRTF, nalar.NALAR_ORDER_SRTF,
                                  nalar.NALAR_ORDER_LPT, 0, 0]):
            say(f"[gpu] wide map/reduce bins pass {i} policy {bits}")
            assert_parity(gpu_run(pol, p, policy=bits), ref[bits], f"bins pass {i}")
            kinds.append(_sort_kind(pol))
    say(f"[gpu] sort kinds {kinds}")
    assert kinds[0] == "tiled" and kinds.count("bin") >= 4, kinds


def test_bin_sort_fallback_and_paths():
    """Bins on the LDS block sweep (1,024-future workflows) and on its HBM
    sweep (8,192-future workflows); a snapshot whose keys all lie past the
    last splitter (every future in one bin: overflow, tiled fallback), then
    equal keys everywhere."""
    lds = _independent(256, 1024, 31)
    hbm = _independent(16, 8192, 32)
    far = lds.copy(deadline_us=lds.deadline_us + (1 << 50))
    flat = _independent(256, 1024, 33, spread=False).copy(est_us=np.full(256 * 1024, 12345, np.int64))
    with nalar.Policy() as pol:
        pol.set_timing(True)
        for i, q in enumerate([lds, lds, lds, far, far, far, lds, hbm, hbm, hbm, flat, flat, flat, lds]):
            say(f"[gpu] bins case {i}: {q.name}")
            check(pol, q, f"bins case {i}")
            say(f"[gpu]   sort {_sort_kind(pol)}")
