"""Reader for the hand-worked fixtures in tests/golden/ (plain text)."""
import os

import numpy as np

from paper_2601_05109_amd.workloads import Problem

GOLDEN_DIR = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load(name: str):
    path = os.path.join(GOLDEN_DIR, name)
    nodes, deadlines, insts, expect = {}, {}, {}, {}
    meta = {}
    with open(path) as fh:
        for raw in fh:
            line = raw.split("#", 1)[0].strip()
            if not line:
                continue
            head, *rest = line.split()
            if head.endswith(":"):
                meta[head[:-1]] = rest[0]
            elif head == "node":
                vid, wf, ty, est, done, loc, deps = rest
                nodes[int(vid)] = (int(wf), int(ty), int(est), int(done), int(loc),
                                   [] if deps == "-" else [int(x) for x in deps.split(",")])
            elif head == "deadline":
                deadlines[int(rest[0])] = int(rest[1])
            elif head == "instance":
                insts[int(rest[0])] = tuple(int(x) for x in rest[1:])
            elif head == "expect":
                expect[rest[0]] = [int(x) for x in rest[1:]]
    N = len(nodes)
    assert sorted(nodes) == list(range(N))
    W = len(deadlines)
    M = len(insts)
    col = lambda i, dt: np.array([nodes[v][i] for v in range(N)], dt)
    deps = [nodes[v][5] for v in range(N)]
    off = np.zeros(N + 1, np.int32)
    off[1:] = np.cumsum([len(d) for d in deps])
    idx = np.array([u for d in deps for u in d], np.int32)
    wf = col(0, np.int32)
    p = Problem(meta["name"], int(meta["now"]), int(meta["mig"]), wf, col(1, np.int32),
                col(2, np.int64), col(3, np.uint8), col(4, np.int32), off, idx,
                np.array([deadlines[w] for w in range(W)], np.int64),
                np.array([insts[i][0] for i in range(M)], np.int32),
                np.array([insts[i][1] for i in range(M)], np.int64),
                np.array([insts[i][2] for i in range(M)], np.int32),
                wf_contiguous=bool(np.all(np.diff(wf) >= 0)))
    return p, expect


def names():
    return sorted(f for f in os.listdir(GOLDEN_DIR) if f.endswith(".txt"))
