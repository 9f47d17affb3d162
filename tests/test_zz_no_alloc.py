"""The pass that allocates nothing (nalar_policy_pass_static) against the
regular pass (nalar_policy_pass) through the C ABI: bit-identical outputs on
two calls in a row, the second with a smaller snapshot, under several policy
variants, with handles sharing the device's array; and the size limit."""
import sys

import numpy as np
import pytest

from paper_2601_05109_amd import workloads as wl

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover - collected on CPU hosts too
    pytest.skip("no GPU", allow_module_level=True)

from paper_2601_05109_amd import nalar  # noqa: E402

FIELDS = ("rem", "order", "slack", "route", "cost")


def say(msg):
    sys.stdout.write(msg + "\n")
    sys.stdout.flush()


def both(pol, p, policy=0, priority=None):
    """One regular pass and one static pass of p on the same handle; the
    host copies of both results."""
    dp = nalar.DeviceProblem.from_host(p)
    pr = None if priority is None else torch.from_numpy(priority).cuda()
    cp = dp.c_struct(policy=policy, priority=pr)
    got = []
    for fn in (nalar.nalar_policy_pass, nalar.nalar_policy_pass_static):
        out = nalar.DeviceResult.alloc(dp.n_nodes)
        for t in (out.order, out.route):  # stale values a pass must overwrite
            t.fill_(-7)
        cr = out.c_struct()
        rc = fn(pol.handle, cp, cr)
        assert rc == nalar.NALAR_OK, (fn.__name__, rc, pol.last_error())
        torch.cuda.synchronize()
        R = int(cr.n_ready)
        got.append({"R": R, "rem": out.rem[:p.n_nodes].cpu().numpy(),
                    **{f: getattr(out, f)[:R].cpu().numpy() for f in FIELDS[1:]}})
    return got


def assert_same(a, b, label):
    assert a["R"] == b["R"], label
    for f in FIELDS:
        np.testing.assert_array_equal(a[f], b[f], err_msg=f"{label}: {f}")


@pytest.mark.parametrize("bits", [0, nalar.NALAR_ORDER_LPT | nalar.NALAR_ROUTE_STATEFUL,
                                  nalar.NALAR_ORDER_SRTF | nalar.NALAR_ROUTE_GREEDY])
def test_static_pass_matches_regular(bits):
    big, small = wl.paper_scale(), wl.tiny()
    with nalar.Policy() as pol:
        for step, p in enumerate((big, small, big, small)):
            say(f"[gpu] static pass step {step}: {p.name} N={p.n_nodes} policy={bits}")
            a, b = both(pol, p, bits)
            assert_same(a, b, f"step {step} {p.name} policy {bits}")


def test_static_pass_levels_and_handles():
    """Priority levels (a level pass in the tiled sort, level groups in the
    buckets), and a second handle on the same device using the same array."""
    p = wl.paper_scale()
    lv = np.random.default_rng(3).integers(0, 16, p.n_workflows).astype(np.uint8)
    with nalar.Policy() as pol, nalar.Policy() as other:
        for i in range(3):
            say(f"[gpu] static levels pass {i}")
            a, b = both(pol, p, 0, lv)
            assert_same(a, b, f"levels pass {i}")
            c, d = both(other, wl.tiny(), nalar.NALAR_ORDER_LPT)
            assert_same(c, d, f"other handle pass {i}")


def test_static_pass_limits():
    """A snapshot beyond the array's limits is rejected with EINVAL (checked on
    the host before anything runs); the largest shape it takes runs."""
    p = wl.windowed(8192)  # 262,144 futures: exactly the node limit
    assert p.n_nodes == nalar.NALAR_STATIC_MAX_NODES
    with nalar.Policy() as pol:
        say("[gpu] static pass at the node limit")
        a, b = both(pol, p)
        assert_same(a, b, "node limit")
        q = wl.windowed(8193)
        dq = nalar.DeviceProblem.from_host(q)
        out = nalar.DeviceResult.alloc(dq.n_nodes)
        rc = nalar.nalar_policy_pass_static(pol.handle, dq.c_struct(), out.c_struct())
        assert rc == nalar.NALAR_EINVAL
        assert "static scratch" in pol.last_error()
