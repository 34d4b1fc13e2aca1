"""CPU checks of the event replay's join state slots (host code only).

An op with two or more direct predecessors (after dropping edges that a
longer path implies) waits on a join word per lane, written when each of
those predecessors is popped and cleared by the last one (Sec. 2's replay
loop releases an op when its last predecessor finishes).  The library may
let joins share a slot when their words are never needed at once.  These
tests take the slots through sim_testing_join_slots and check, on schedules
of the oracle, that joins sharing a slot are never open together: in the pop
order of the replay (ready time, priority, id), every predecessor pop of one
comes before every predecessor pop of the other.  The schedules use random
durations, so a slot shared on a wrong condition shows up as an overlap.
"""
import numpy as np
import pytest

import oracle
from paper_2002_06790_amd import workloads as W

mlsim = pytest.importorskip("paper_2002_06790_amd")


@pytest.fixture(scope="module")
def lib():
    import os
    if not os.path.exists(mlsim.LIB_PATH):
        pytest.skip("libmlsim.so is not built")
    return mlsim


def direct_preds(ptr, idx, n):
    """Predecessors of each op that no longer path implies (brute force on
    ancestor sets held as Python integers)."""
    preds = [set() for _ in range(n)]
    for u in range(n):
        for v in idx[ptr[u]:ptr[u + 1]].tolist():
            preds[v].add(u)
    succ = [[] for _ in range(n)]
    cnt = [len(p) for p in preds]
    for v in range(n):
        for u in preds[v]:
            succ[u].append(v)
    order = [v for v in range(n) if cnt[v] == 0]
    for u in order:
        for v in succ[u]:
            cnt[v] -= 1
            if cnt[v] == 0:
                order.append(v)
    assert len(order) == n
    anc = [0] * n  # proper ancestors
    for v in order:
        a = 0
        for u in preds[v]:
            a |= anc[u] | (1 << u)
        anc[v] = a
    red = []
    for v in range(n):
        # u is implied when it is an ancestor of another predecessor of v
        others = 0
        for u in preds[v]:
            others |= anc[u]
        red.append(sorted(u for u in preds[v] if not (others >> u) & 1))
    return red


def check_slots(lib, ptr, idx, res, R, prio, dur):
    n = dur.shape[0]
    slot_of, n_slots = lib.join_slots(ptr, idx, res, R, prio=prio)
    red = direct_preds(ptr, idx, n)
    joins = {}  # (slot, predecessor set) -> one join (ops with the same set share it)
    for v in range(n):
        if len(red[v]) >= 2:
            assert 0 <= slot_of[v] < n_slots, f"op {v} waits on a join"
            joins.setdefault((int(slot_of[v]), tuple(red[v])), v)
        else:
            assert slot_of[v] == -1, f"op {v} has {len(red[v])} direct predecessors"
    assert n_slots <= len(joins)
    _, fin, st = oracle.run_batch(ptr, idx, res, R, dur, prio=prio)
    assert (st == 0).all()
    pr = np.arange(n) if prio is None else np.asarray(prio)
    for s in range(dur.shape[1]):
        f = fin[:, s].astype(np.int64)
        ready = np.array([max((f[u] for u in red[v]), default=0) for v in range(n)], np.int64)
        pos = np.empty(n, np.int64)
        pos[np.lexsort((np.arange(n), pr, ready))] = np.arange(n)
        by_slot = {}
        for (sl, ps) in joins:
            p = pos[list(ps)]
            by_slot.setdefault(sl, []).append((int(p.min()), int(p.max())))
        for sl, iv in by_slot.items():
            iv.sort()
            for (a0, a1), (b0, b1) in zip(iv, iv[1:]):
                assert a1 < b0, f"slot {sl}: joins open together in scenario {s}"
    return len(joins), n_slots


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_workload_slots(lib, k):
    w = W.make_config(k, n_scen=4)
    dur = w.durations()
    nj, ns = check_slots(lib, w.succ_ptr, w.succ_idx, w.op_res, w.n_res, w.prio, dur)
    print(f"{w.name}: {nj} joins in {ns} slots", flush=True)
    if w.name == "random-layered":
        # 200 levels fed by the previous level: a join's slot is free again a
        # few levels later
        assert ns * 4 < nj


def test_random_graph_slots(lib):
    """Random DAGs (duplicate edges, priorities, several components)."""
    rng = np.random.default_rng(2002)
    for case in range(60):
        n = int(rng.choice([2, 5, 17, 40, 120, 300]))
        R = int(rng.integers(1, 6))
        ptr, idx, res, pr = W.random_dag(n, R, float(rng.uniform(0.02, 0.5)), rng,
                                         with_prio=bool(rng.integers(2)), dup_edges=bool(rng.integers(2)))
        dur = W.random_durations(n, 6, 1, 1000, rng)
        check_slots(lib, ptr, idx, res, R, pr, dur)


def test_layered_chain_reuses_slots(lib):
    """Levels of 4 ops, each op fed by every op of the previous level: the
    ops of a level share one join (a barrier), and each level's join can take
    the slot of the previous level's (its predecessors are the ops that join
    released), so one slot serves them all."""
    L, width = 30, 4
    n = L * width
    succ = [[] for _ in range(n)]
    for l in range(L - 1):
        for a in range(width):
            succ[l * width + a] = [(l + 1) * width + b for b in range(width)]
    ptr = np.zeros(n + 1, np.int64)
    ptr[1:] = np.cumsum([len(x) for x in succ])
    idx = np.array([x for s in succ for x in s], np.int32)
    dur = W.random_durations(n, 8, 1, 1000, np.random.default_rng(3))
    nj, ns = check_slots(lib, ptr, idx, np.zeros(n, np.int32), 1, None, dur)
    assert nj == L - 1 and ns == 1


def test_slot_errors(lib):
    ptr = np.array([0, 1, 0], np.int64)
    with pytest.raises(mlsim.SimError):
        lib.join_slots(ptr, np.array([1], np.int32), np.zeros(2, np.int32), 1)
    with pytest.raises(mlsim.SimError) as e:  # a cycle
        lib.join_slots(np.array([0, 1, 2], np.int64), np.array([1, 0], np.int32), np.zeros(2, np.int32), 1)
    assert e.value.code == mlsim.SIM_E_CYCLE
    slot_of, ns = lib.join_slots(np.zeros(1, np.int64), np.zeros(0, np.int32), np.zeros(0, np.int32), 1)
    assert slot_of.size == 0 and ns == 0
