"""Loader for the hand-derived worked examples under tests/golden/."""
from __future__ import annotations

import glob
import os

import numpy as np

GOLDEN_DIR = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load(path):
    ops, kv = [], {}
    n_res = None
    for line in open(path):
        line = line.split("#", 1)[0].split()
        if not line:
            continue
        if line[0] == "resources":
            n_res = int(line[1])
        elif line[0] == "op":
            vid, res, dur, prio = int(line[1]), int(line[2]), int(line[3]), line[4]
            preds = [] if line[5:] == ["-"] else [int(x) for x in line[5:]]
            assert vid == len(ops)
            ops.append((res, dur, None if prio == "-" else int(prio), preds))
        else:
            kv[line[0]] = [int(x) for x in line[1:]]
    n = len(ops)
    succ = [[] for _ in range(n)]
    for v, (_, _, _, preds) in enumerate(ops):
        for u in preds:
            succ[u].append(v)
    ptr = np.zeros(n + 1, np.int64)
    ptr[1:] = np.cumsum([len(s) for s in succ])
    idx = np.array([w for s in succ for w in s], np.int32)
    res = np.array([o[0] for o in ops], np.int32)
    dur = np.array([[o[1]] for o in ops], np.int32)
    prio = None
    if any(o[2] is not None for o in ops):
        prio = np.array([o[2] if o[2] is not None else v for v, o in enumerate(ops)], np.int32)
    return dict(name=os.path.basename(path), n=n, n_res=n_res, succ_ptr=ptr, succ_idx=idx,
                op_res=res, prio=prio, dur=dur, expect=kv)


def all_goldens():
    """The worked examples of the plain replay (exclusive devices)."""
    return [load(p) for p in sorted(glob.glob(os.path.join(GOLDEN_DIR, "example_*.txt")))]


def share_goldens():
    """The worked examples of the replay with bandwidth sharing (a "shared"
    line gives each resource's flag)."""
    return [load(p) for p in sorted(glob.glob(os.path.join(GOLDEN_DIR, "share_*.txt")))]
