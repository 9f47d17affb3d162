"""The seeded generators produce the stated shapes and distributions."""
import numpy as np
import pytest

from paper_2601_05109_amd import workloads as wl


@pytest.mark.parametrize("name,N,W,M,K", [("tiny", 2048, 64, 16, 4), ("paper-scale", 131072, 4096, 64, 8),
                                         ("deep-chains", 524288, 1024, 128, 8),
                                         ("wide-mapreduce", 1049088, 256, 256, 8)])
def test_shapes_and_ranges(name, N, W, M, K):
    p = wl.WORKLOADS[name]()
    p.check_dtypes()
    assert (p.n_nodes, p.n_workflows, p.n_instances) == (N, W, M)
    assert p.wf_contiguous and np.all(np.diff(p.wf) >= 0)
    assert p.type.min() >= 0 and p.type.max() < K and p.inst_type.max() < K
    assert p.est_us.min() >= 1 and p.est_us.max() <= 1 << 40
    assert p.loc.min() >= -1 and p.loc.max() < M
    assert 0.45 < (p.loc >= 0).mean() < 0.55
    assert p.inst_speed_permille.min() >= 500 and p.inst_speed_permille.max() <= 2000
    assert p.inst_load_us.min() >= 0 and p.inst_load_us.max() <= 2_000_000
    d = p.deadline_us - p.now_us
    assert d.min() >= 2_000_000 and d.max() <= 20_000_000
    # parents precede children inside the same workflow
    child = np.repeat(np.arange(N), np.diff(p.dep_off.astype(np.int64)))
    assert np.all(p.dep_idx < child) and np.all(p.wf[p.dep_idx] == p.wf[child])


def test_windowed_parents():
    p = wl.paper_scale()
    N = p.n_nodes
    child = np.repeat(np.arange(N), np.diff(p.dep_off.astype(np.int64)))
    gap = child - p.dep_idx
    assert gap.min() >= 1 and gap.max() <= 8
    cnt = np.diff(p.dep_off)
    assert cnt.max() <= 3 and np.all(cnt[::32] == 0) and np.all(cnt.reshape(-1, 32)[:, 1:] >= 1)
    assert abs(cnt.mean() - 1.42) < 0.05           # 1 + E[min(Poisson(0.5), 2)]
    assert np.all(p.done.reshape(-1, 32)[:, :9] == 1) and np.all(p.done.reshape(-1, 32)[:, 9:] == 0)
    llm = p.type < 2
    assert abs(np.median(p.est_us[llm]) / 800_000 - 1) < 0.03
    assert abs(np.median(p.est_us[~llm]) / 50_000 - 1) < 0.03


def test_deterministic():
    a, b = wl.paper_scale(), wl.paper_scale()
    assert a.digest() == b.digest()
    assert wl.paper_scale(seed=5).digest() != a.digest()


def test_dynamic_stream_first_steps():
    it = wl.dynamic_stream(steps=3)
    p0 = next(it)
    assert p0.n_nodes == 1_049_088 and p0.wf_contiguous
    n0 = p0.n_nodes
    p1 = next(it)
    assert p1.n_nodes > n0 and not p1.wf_contiguous
    # appended children have exactly one dependency, in their workflow
    new = np.arange(n0, p1.n_nodes)
    assert np.all(np.diff(p1.dep_off[n0:].astype(np.int64)) == 1)
    par = p1.dep_idx[p1.dep_off[n0]:]
    assert np.all(p1.wf[new] == p1.wf[par]) and np.all(p1.done[new] == 0)
    assert 0 < int(p1.done.sum()) - 256 <= 1_048_576 // 100
