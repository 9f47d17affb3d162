"""CPU-side checks of the HIP library: it loads, exports every function the
public header declares, the binding refuses to run without it, and the exact
division used by the routing scorer matches integer division (host build of the
same helper).  Nothing here launches GPU work."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "nalar_policy.h")
HEADERS = [os.path.join(ROOT, "include", f) for f in sorted(os.listdir(os.path.join(ROOT, "include")))
           if f.endswith(".h")]
LIB = os.path.join(ROOT, "paper_2601_05109_amd", "libnalar_policy.so")


def declared_functions():
    names = set()
    for h in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(nalar_(?:policy|store)_\w+)\s*\(", text))
    return sorted(names)


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        from paper_2601_05109_amd import build
        build.build()
    return ctypes.CDLL(LIB)


def test_header_declares_the_abi():
    names = declared_functions()
    for required in ("nalar_policy_create", "nalar_policy_pass", "nalar_policy_destroy",
                     "nalar_policy_last_error", "nalar_store_create", "nalar_store_append",
                     "nalar_store_complete", "nalar_store_pass"):
        assert required in names


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), f"{name} not exported"


def test_binding_names_match_header():
    from paper_2601_05109_amd import nalar
    assert sorted(nalar.EXPORTED) == declared_functions()
    for name in nalar.EXPORTED:
        assert callable(getattr(nalar, name))


def test_struct_layouts_match_header():
    """Sizes and offsets of the ctypes mirrors equal the C structs (compiled
    with the host compiler against the header)."""
    from paper_2601_05109_amd import nalar
    src = r'''
#include <stdio.h>
#include <stddef.h>
#include "nalar_policy.h"
int main(void) {
  printf("%zu %zu %zu\n", sizeof(nalar_policy_config), sizeof(nalar_problem), sizeof(nalar_result));
  printf("%zu %zu %zu %zu %zu\n", offsetof(nalar_problem, flags), offsetof(nalar_problem, wf),
         offsetof(nalar_problem, inst_speed_permille), offsetof(nalar_problem, wf_priority),
         offsetof(nalar_result, n_ready));
  printf("%zu\n", offsetof(nalar_policy_config, reserve_workflows));
  printf("%zu %zu %zu %zu %zu\n", offsetof(nalar_problem, inst_weight), sizeof(nalar_view),
         offsetof(nalar_view, n_order), sizeof(nalar_decisions), offsetof(nalar_decisions, rank));
  return 0;
}
'''
    import tempfile
    with tempfile.TemporaryDirectory() as d:
        c = os.path.join(d, "l.c")
        open(c, "w").write(src)
        exe = os.path.join(d, "l")
        subprocess.run(["gcc", "-I", os.path.dirname(HEADER), c, "-o", exe], check=True)
        out = subprocess.run([exe], capture_output=True, text=True, check=True).stdout.split()
    got = list(map(int, out))
    P, C, R = nalar.NalarProblem, nalar.NalarPolicyConfig, nalar.NalarResult
    V, D = nalar.NalarView, nalar.NalarDecisions
    assert got == [ctypes.sizeof(C), ctypes.sizeof(P), ctypes.sizeof(R), P.flags.offset,
                   P.wf.offset, P.inst_speed_permille.offset, P.wf_priority.offset, R.n_ready.offset,
                   C.reserve_workflows.offset, P.inst_weight.offset, ctypes.sizeof(V),
                   V.n_order.offset, ctypes.sizeof(D), D.rank.offset]


def test_binding_fails_loudly_without_library(tmp_path):
    from paper_2601_05109_amd import nalar
    saved = nalar._lib
    nalar._lib = None
    try:
        with pytest.raises(RuntimeError, match="missing"):
            nalar.load_library(str(tmp_path / "absent.so"))
    finally:
        nalar._lib = saved


def test_exact_division_helper(tmp_path):
    exe = tmp_path / "floordiv_check"
    hipcc = "/opt/rocm/bin/hipcc"
    subprocess.run([hipcc, "-O2", "-std=c++17", "-I", os.path.join(ROOT, "include"),
                    "-I", os.path.join(ROOT, "paper_2601_05109_amd", "csrc"),
                    os.path.join(ROOT, "tests", "floordiv_check.cpp"), "-o", str(exe)],
                   check=True, capture_output=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stdout
    assert "mismatches 0" in r.stdout


def test_routing_scorer(tmp_path):
    """The routing scorer against a plain integer argmin on random, tied and
    near-tied instance tables, loads near 2^60, speeds near 2^31 and
    estimates near 2^40."""
    exe = tmp_path / "routing_check"
    hipcc = "/opt/rocm/bin/hipcc"
    subprocess.run([hipcc, "-O2", "-std=c++17", "-I", os.path.join(ROOT, "include"),
                    "-I", os.path.join(ROOT, "paper_2601_05109_amd", "csrc"),
                    os.path.join(ROOT, "tests", "routing_check.cpp"), "-o", str(exe)],
                   check=True, capture_output=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stdout
    assert "mismatches 0" in r.stdout


def test_kernels_keep_their_registers(tmp_path):
    """No kernel spills to scratch memory beyond a small bound: a spill that
    grows (the block sweep runs at the 128-register limit of 1024-thread
    workgroups) turns into per-lane scratch traffic to HBM and slows the pass
    several times over.  Resource usage as the compiler reports it for the
    library's own build flags."""
    from paper_2601_05109_amd import build
    csrc = os.path.join(ROOT, "paper_2601_05109_amd", "csrc")
    worst = {}
    for src in sorted(f for f in os.listdir(csrc) if f.endswith(".hip")):
        r = subprocess.run([build.HIPCC, *build.FLAGS, "-c", os.path.join(csrc, src), "-o",
                            str(tmp_path / (src + ".o")), "-Rpass-analysis=kernel-resource-usage"],
                           capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        name = None
        for line in r.stderr.splitlines():
            m = re.search(r"Function Name: (\S+)", line)
            if m:
                name = m.group(1)
            m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
            if m and name:
                worst[name] = int(m.group(1))
    assert worst, "no kernel resource remarks"
    over = {k: v for k, v in worst.items() if v > 96}
    assert not over, f"kernels spilling to scratch: {over}"
