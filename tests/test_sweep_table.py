"""CPU checks of the max-plus sweep tables the library builds (host code only).

The library compiles a graph into a table of records that the sweep kernel
visits in order: dist(record) = duration (0 for a barrier record) + max over
its predecessor slots, written to its own slot.  The table builder chooses
barrier records for shared predecessor sets, a topological order and a slot
per live value.  These tests take the table through sim_testing_sweep_table
(no device is used), evaluate it with the plain interpreter below, and compare
the result with the oracle: the critical path (Sec. 1: the bound the
bottleneck analysis starts from) and the static-order replay (Sec. 2 devices
with a fixed queue order).  A slot reused while its value is still needed, a
wrong barrier set or an order that is not topological changes the numbers.
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


def interpret(rec, plist, slots, dur):
    """Evaluate a sweep table on durations dur [n_ops, S]: returns dist of
    every op [n_ops, S] (its finish time in a static-order replay)."""
    n, S = dur.shape
    val = np.zeros((slots, S), np.int64)
    dist = np.full((n, S), -1, np.int64)
    written = np.zeros(n, np.int64)
    zslot = slots - 2
    for row, slot, npred, pbeg, p0, p1, p2, p3 in rec.tolist():
        preds = [p0, p1, p2, p3][:npred] if npred <= 4 else plist[pbeg:pbeg + npred].tolist()
        if npred <= 4:
            assert all(p == zslot for p in [p0, p1, p2, p3][npred:]), "unused entries name the zero slot"
        assert 0 <= slot < slots and slot != zslot, "a record writes a real slot"
        best = val[preds].max(axis=0) if preds else np.zeros(S, np.int64)
        x = best + (dur[row].astype(np.int64) if row >= 0 else 0)
        val[slot] = x
        if row >= 0:
            dist[row] = x
            written[row] += 1
    assert (written == 1).all(), "every op is swept exactly once"
    assert (val[zslot] == 0).all()
    return dist


def check_cp(lib, ptr, idx, res, R, dur, prio=None):
    rec, plist, slots = lib.sweep_table(ptr, idx, res, R, prio=prio)
    dist = interpret(rec, plist, slots, dur)
    ocp, _ = oracle.critical_path(ptr, idx, dur.shape[0], dur)
    assert np.array_equal(dist.max(axis=0) if dur.shape[0] else np.zeros(dur.shape[1]), ocp)
    return rec, slots


def check_static(lib, ptr, idx, res, R, order, dur, prio=None):
    rec, plist, slots = lib.sweep_table(ptr, idx, res, R, prio=prio, order=order)
    dist = interpret(rec, plist, slots, dur)
    omk, ofin, ost = oracle.static_run(ptr, idx, res, R, order, dur)
    assert ost[0] == 0 and set(np.unique(ost)) <= {0, 4}  # durations >= 1: only overflow can flag
    ok = ost == 0
    assert np.array_equal(dist[:, ok], ofin[:, ok]), "finish times differ"
    assert np.array_equal(dist.max(axis=0)[ok], omk[ok])
    # a scenario whose run order (made for scenario 0) overflows: its exact
    # finish times exceed INT32_MAX there and nowhere else
    assert np.array_equal(dist.max(axis=0) > 2**31 - 1, ~ok)
    return rec, slots


def event_order(dur0, fin0):
    n = dur0.size
    return np.lexsort((np.arange(n), fin0.astype(np.int64) - dur0)).astype(np.int32)


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_workload_tables(lib, k):
    """Critical-path and static-order tables of every workload (the static
    order: the event replay's run order in scenario 0)."""
    w = W.make_config(k, n_scen=24)
    dur = w.durations()
    rec, slots = check_cp(lib, w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur, prio=w.prio)
    place = w.placement()
    res = w.op_res if place is None else place[:, 0].astype(np.int32)
    _, f0, _ = oracle.run_batch(w.succ_ptr, w.succ_idx, res, w.n_res, dur[:, :1], prio=w.prio)
    order = event_order(dur[:, 0], f0[:, 0])
    srec, sslots = check_static(lib, w.succ_ptr, w.succ_idx, res, w.n_res, order, dur, prio=w.prio)
    print(f"{w.name}: critical-path table {len(rec)} records, {slots} slots; "
          f"static table {len(srec)} records, {sslots} slots", flush=True)
    if w.name == "bert-large-ps":
        # the pushes -> pulls all-to-all: one barrier per bucket, few live values
        assert (rec[:, 0] < 0).sum() == 25 and slots <= 40
        assert (srec[:, 0] < 0).sum() == 25 and sslots <= 80


def fan_graph(m, k, chain):
    n = m + k + k * chain
    succ = [[] for _ in range(n)]
    for s in range(m):
        succ[s] = list(range(m, m + k))
    for j in range(k):
        prev = m + j
        for c in range(chain):
            v = m + k + j * chain + c
            succ[prev].append(v)
            prev = v
    ptr = np.zeros(n + 1, np.int64)
    ptr[1:] = np.cumsum([len(x) for x in succ])
    return ptr, np.array([x for s in succ for x in s], np.int32), n


@pytest.mark.parametrize("m,k,chain", [(6, 6, 2), (5, 4, 1), (3, 3, 1), (8, 3, 2)])
def test_fan_graph_tables_use_barriers(lib, m, k, chain):
    """m sources feeding k joins: the builder takes the barrier table, for the
    critical path and for a static replay with every op on its own
    resource."""
    ptr, idx, n = fan_graph(m, k, chain)
    dur = W.random_durations(n, 40, 1, 1000, np.random.default_rng(m * 100 + k))
    rec, _ = check_cp(lib, ptr, idx, np.zeros(n, np.int32), 1, dur)
    assert (rec[:, 0] < 0).sum() == 1
    srec, _ = check_static(lib, ptr, idx, np.arange(n, dtype=np.int32), n, np.arange(n, dtype=np.int32), dur)
    assert (srec[:, 0] < 0).sum() == 1


def test_static_shared_sets_beside_device_edges(lib):
    """Joins sharing a predecessor set on one resource: each also waits for
    the previous join on its resource, and the barrier is still shared."""
    m, k = 5, 6
    ptr, idx, n = fan_graph(m, k, 0)
    res = np.concatenate([np.arange(m), np.full(k, m)]).astype(np.int32)
    order = np.arange(n, dtype=np.int32)
    dur = W.random_durations(n, 40, 1, 1000, np.random.default_rng(9))
    srec, _ = check_static(lib, ptr, idx, res, m + 1, order, dur)
    assert (srec[:, 0] < 0).sum() == 1


def test_random_graph_tables(lib):
    """Random DAGs (duplicate edges, priorities, long predecessor lists,
    several components) and random valid run orders."""
    rng = np.random.default_rng(20020679)
    for case in range(40):
        n = int(rng.choice([1, 2, 5, 16, 17, 40, 120]))
        R = int(rng.integers(1, 6))
        ptr, idx, res, pr = W.random_dag(n, R, float(rng.uniform(0.02, 0.6)), rng,
                                         with_prio=bool(rng.integers(2)), dup_edges=bool(rng.integers(2)))
        dur = W.random_durations(n, 8, 1, 1000, rng)
        check_cp(lib, ptr, idx, res, R, dur, prio=pr)
        # a random topological order (Kahn with random choices) as the run order
        cnt = np.zeros(n, np.int64)  # predecessors, duplicate edges counted once
        for u in range(n):
            for v in np.unique(idx[ptr[u]:ptr[u + 1]]):
                cnt[v] += 1
        ready = [v for v in range(n) if cnt[v] == 0]
        order = []
        while ready:
            v = ready.pop(int(rng.integers(len(ready))))
            order.append(v)
            for x in np.unique(idx[ptr[v]:ptr[v + 1]]):
                cnt[x] -= 1
                if cnt[x] == 0:
                    ready.append(int(x))
        check_static(lib, ptr, idx, res, R, np.array(order, np.int32), dur, prio=pr)


def test_table_errors(lib):
    ptr = np.array([0, 1, 2, 2], np.int64)
    idx = np.array([1, 2], np.int32)
    res = np.zeros(3, np.int32)
    for bad, code in (([0, 0, 1], mlsim.SIM_E_INVAL), ([0, 1, 3], mlsim.SIM_E_INVAL),
                      ([1, 0, 2], mlsim.SIM_E_CYCLE)):
        with pytest.raises(mlsim.SimError) as e:
            lib.sweep_table(ptr, idx, res, 1, order=np.array(bad, np.int32))
        assert e.value.code == code
    with pytest.raises(mlsim.SimError) as e:
        lib.sweep_table(ptr, np.array([1, 3], np.int32), res, 1)
    assert e.value.code == mlsim.SIM_E_RANGE
    with pytest.raises(mlsim.SimError) as e:  # a cycle in the graph itself
        lib.sweep_table(np.array([0, 1, 2], np.int64), np.array([1, 0], np.int32), np.zeros(2, np.int32), 1)
    assert e.value.code == mlsim.SIM_E_CYCLE
    rec, plist, slots = lib.sweep_table(np.zeros(1, np.int64), np.zeros(0, np.int32), np.zeros(0, np.int32), 1)
    assert rec.shape == (0, 8)
