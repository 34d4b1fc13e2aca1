"""Pins of the CPU oracle against what the paper's model and mathematics fix.

The oracle (oracle/oracle.c) replays the simulation loop of Sec. 2
("Dataflow based simulation").  Nothing here re-runs the oracle's own code to
check it: the pins are hand-derived worked examples, closed forms, bounds,
structural invariants of a FIFO device, metamorphic relations, a library
shortest-path routine, and two independent brute-force replays (tests/brute.py).
"""
import os

import math

import numpy as np
import pytest
import scipy.sparse
import scipy.sparse.csgraph

import oracle
import brute
import goldens
from paper_2002_06790_amd.workloads import random_dag, random_durations


# ------------------------------------------------------------------ helpers

def oracle_run(library, *a, **kw):
    return oracle.run_batch(*a, library=library, **kw)


def oracle_cp(library, *a, **kw):
    return oracle.critical_path(*a, library=library, **kw)


def run(g, dur, library=None, **kw):
    return oracle.run_batch(g["succ_ptr"], g["succ_idx"], g["op_res"], g["n_res"], dur,
                            prio=g.get("prio"), library=library, **kw)


def rand_graph(rng, n, n_res, p, prio=False, dup=False, shuffle=True):
    ptr, idx, res, pr = random_dag(n, n_res, p, rng, shuffle_ids=shuffle, with_prio=prio,
                                   dup_edges=dup)
    return dict(n=n, n_res=n_res, succ_ptr=ptr, succ_idx=idx, op_res=res, prio=pr)


def preds(g):
    return brute.preds_of(g["n"], g["succ_ptr"], g["succ_idx"])


def schedule_checks(g, dur_col, fin_col, span):
    """Structural invariants of one scenario's schedule (FIFO devices)."""
    n = g["n"]
    P = preds(g)
    prio = g["prio"] if g["prio"] is not None else np.arange(n)
    d = dur_col.astype(np.int64)
    f = fin_col.astype(np.int64)
    start = f - d
    ready = np.array([max([f[u] for u in P[v]], default=0) for v in range(n)])
    assert (start >= ready).all(), "an op starts before its inputs are ready"
    assert span == (f.max() if n else 0)
    for r in range(g["n_res"]):
        ops = [v for v in range(n) if g["op_res"][v] == r]
        ops.sort(key=lambda v: start[v])
        prev_fin = 0
        for k, v in enumerate(ops):
            assert start[v] >= prev_fin, "two ops overlap on one device"
            # non-delay: a device never idles while its queue is non-empty
            assert start[v] == max(ready[v], prev_fin)
            prev_fin = f[v]
            if k:
                u = ops[k - 1]
                assert (ready[u], prio[u], u) < (ready[v], prio[v], v), "device not FIFO by key"
    return start, ready


# ------------------------------------------------------------------ goldens

@pytest.mark.parametrize("g", goldens.all_goldens(), ids=lambda g: g["name"])
def test_worked_examples(g, library):
    ex = g["expect"]
    mk, fin, st = run(g, g["dur"], library=library)
    assert st.tolist() == [0]
    assert fin[:, 0].tolist() == ex["finish"]
    assert mk.tolist() == ex["makespan"]
    if "cp_len" in ex:
        cp, path = oracle_cp(library, g["succ_ptr"], g["succ_idx"], g["n"], g["dur"], 0)
        assert cp.tolist() == ex["cp_len"]
        assert path.tolist() == ex["cp_path"]
    if "dur2" in ex:
        d2 = np.array(ex["dur2"], np.int32)[:, None]
        mk2, fin2, _ = run(g, d2, library=library)
        assert fin2[:, 0].tolist() == ex["finish2"]
        assert mk2.tolist() == ex["makespan2"]


@pytest.mark.parametrize("g", goldens.all_goldens(), ids=lambda g: g["name"])
def test_worked_examples_tick_sim(g, library):
    """The brute-force tick simulator reproduces the hand-derived values."""
    fin = brute.tick_sim(g["n"], g["n_res"], g["succ_ptr"], g["succ_idx"], g["op_res"],
                         g["dur"][:, 0], g["prio"])
    assert fin == g["expect"]["finish"]


# -------------------------------------------------------------- closed forms

def test_no_edges_prefix_sums(library):
    """Without edges each device runs its ops in (priority, id) order back to back."""
    rng = np.random.default_rng(1)
    for _ in range(30):
        n, R = int(rng.integers(1, 40)), int(rng.integers(1, 5))
        g = rand_graph(rng, n, R, 0.0, prio=bool(rng.integers(2)))
        dur = random_durations(n, 3, 1, 50, rng)
        mk, fin, _ = run(g, dur, library=library)
        prio = g["prio"] if g["prio"] is not None else np.arange(n)
        for s in range(3):
            expect = np.zeros(n, np.int64)
            for r in range(R):
                ops = sorted((v for v in range(n) if g["op_res"][v] == r), key=lambda v: (prio[v], v))
                expect[ops] = np.cumsum(dur[ops, s])
            assert (fin[:, s] == expect).all()
            assert mk[s] == expect.max()


def test_chain_cumulative_sums(library):
    """A chain runs back to back whatever its devices: finish = prefix sums."""
    rng = np.random.default_rng(2)
    for _ in range(30):
        n, R = int(rng.integers(1, 60)), int(rng.integers(1, 6))
        order = rng.permutation(n)
        succ = [[] for _ in range(n)]
        for a, b in zip(order, order[1:]):
            succ[a].append(int(b))
        ptr = np.zeros(n + 1, np.int64)
        ptr[1:] = np.cumsum([len(s) for s in succ])
        idx = np.array([w for s in succ for w in s], np.int32)
        res = rng.integers(0, R, n).astype(np.int32)
        dur = random_durations(n, 4, 1, 1000, rng)
        mk, fin, _ = oracle_run(library, ptr, idx, res, R, dur)
        assert (fin[order] == np.cumsum(dur[order], axis=0)).all()
        assert (mk == dur.sum(0)).all()


def test_single_device_makespan_is_total_work(library):
    """With one device it never idles: makespan = sum of durations."""
    rng = np.random.default_rng(3)
    for _ in range(30):
        n = int(rng.integers(1, 80))
        g = rand_graph(rng, n, 1, float(rng.uniform(0, 0.3)), prio=True)
        dur = random_durations(n, 5, 1, 100, rng)
        mk, _, _ = run(g, dur, library=library)
        assert (mk == dur.sum(0)).all()


def longest_path_scipy(g, dur_col):
    """Longest path via scipy's Bellman-Ford on negated node weights."""
    n = g["n"]
    src, dst, w = [], [], []
    ptr, idx = g["succ_ptr"], g["succ_idx"]
    seen = set()
    for u in range(n):
        for e in range(ptr[u], ptr[u + 1]):
            v = int(idx[e])
            if (u, v) not in seen:
                seen.add((u, v))
                src.append(u), dst.append(v), w.append(-float(dur_col[v]))
    for v in range(n):  # virtual source n
        src.append(n), dst.append(v), w.append(-float(dur_col[v]))
    A = scipy.sparse.csr_matrix((w, (src, dst)), shape=(n + 1, n + 1))
    D = scipy.sparse.csgraph.shortest_path(A, method="BF", directed=True, indices=n)
    return -D[:n]


def test_unlimited_devices_equals_longest_path(library):
    """One device per op: finish = longest path to the op; makespan = critical path."""
    rng = np.random.default_rng(4)
    for _ in range(25):
        n = int(rng.integers(1, 60))
        g = rand_graph(rng, n, 1, float(rng.uniform(0, 0.25)))
        g["n_res"] = n
        g["op_res"] = np.arange(n, dtype=np.int32)
        dur = random_durations(n, 3, 1, 1000, rng)
        mk, fin, _ = run(g, dur, library=library)
        cp, _ = oracle_cp(library, g["succ_ptr"], g["succ_idx"], n, dur)
        for s in range(3):
            dist = longest_path_scipy(g, dur[:, s])
            assert (fin[:, s] == dist).all()
            assert mk[s] == cp[s] == dist.max()


# -------------------------------------------------------------- brute force

def test_matches_tick_simulator(library):
    rng = np.random.default_rng(5)
    for _ in range(150):
        n, R = int(rng.integers(1, 9)), int(rng.integers(1, 4))
        g = rand_graph(rng, n, R, float(rng.uniform(0, 0.6)), prio=bool(rng.integers(2)),
                       dup=bool(rng.integers(2)))
        dur = random_durations(n, 2, 1, 6, rng)
        mk, fin, _ = run(g, dur, library=library)
        for s in range(2):
            ref = brute.tick_sim(n, R, g["succ_ptr"], g["succ_idx"], g["op_res"], dur[:, s], g["prio"])
            assert fin[:, s].tolist() == ref
            assert mk[s] == max(ref)


def test_unique_fifo_consistent_order(library):
    """Exactly one per-device order is FIFO by (ready, prio, id); it is the oracle's."""
    rng = np.random.default_rng(6)
    for _ in range(60):
        n, R = int(rng.integers(1, 7)), int(rng.integers(1, 3))
        g = rand_graph(rng, n, R, float(rng.uniform(0, 0.6)), prio=bool(rng.integers(2)))
        dur = random_durations(n, 1, 1, 6, rng)
        _, fin, _ = run(g, dur, library=library)
        found = brute.enumerate_orders(n, R, g["succ_ptr"], g["succ_idx"], g["op_res"], dur[:, 0],
                                       g["prio"])
        assert len(found) == 1
        assert found[0] == fin[:, 0].tolist()


# --------------------------------------------------------------- invariants

def test_bounds_and_structure_random(library):
    rng = np.random.default_rng(7)
    for _ in range(30):
        n, R = int(rng.integers(1, 300)), int(rng.integers(1, 12))
        g = rand_graph(rng, n, R, float(rng.uniform(0, 8.0 / max(n, 1))), prio=bool(rng.integers(2)))
        dur = random_durations(n, 3, 1, 10_000, rng)
        mk, fin, st = run(g, dur, library=library)
        cp, _ = oracle_cp(library, g["succ_ptr"], g["succ_idx"], n, dur)
        assert (st == 0).all()
        for s in range(3):
            schedule_checks(g, dur[:, s], fin[:, s], mk[s])
            busy = np.bincount(g["op_res"], weights=dur[:, s], minlength=R).max()
            assert max(cp[s], busy) <= mk[s] <= dur[:, s].sum()


def test_scaling_durations_scales_times(library):
    rng = np.random.default_rng(8)
    for _ in range(15):
        n, R = int(rng.integers(1, 100)), int(rng.integers(1, 6))
        g = rand_graph(rng, n, R, 0.05, prio=True)
        dur = random_durations(n, 3, 1, 100, rng)
        k = int(rng.integers(2, 50))
        mk, fin, _ = run(g, dur, library=library)
        mk2, fin2, _ = run(g, dur * k, library=library)
        assert (mk2 == k * mk).all() and (fin2 == k * fin).all()


def test_relabel_resources_and_shuffle_columns(library):
    rng = np.random.default_rng(9)
    for _ in range(15):
        n, R = int(rng.integers(1, 100)), int(rng.integers(1, 8))
        g = rand_graph(rng, n, R, 0.05)
        dur = random_durations(n, 16, 1, 100, rng)
        mk, fin, _ = run(g, dur, library=library)
        perm = rng.permutation(R).astype(np.int32)
        g2 = dict(g, op_res=perm[g["op_res"]])
        cols = rng.permutation(16)
        mk2, fin2, _ = run(g2, dur[:, cols], library=library)
        assert (mk2 == mk[cols]).all() and (fin2 == fin[:, cols]).all()


def test_relabel_ops_with_equivalent_priorities(library):
    """Renumbering ops while keeping their (priority, id) order keeps the schedule."""
    rng = np.random.default_rng(10)
    for _ in range(15):
        n, R = int(rng.integers(2, 80)), int(rng.integers(1, 5))
        g = rand_graph(rng, n, R, 0.08, prio=True)
        dur = random_durations(n, 4, 1, 8, rng)  # small values: many ties
        mk, fin, _ = run(g, dur, library=library)
        pi = rng.permutation(n)  # old id -> new id
        rank = np.empty(n, np.int32)
        rank[np.lexsort((np.arange(n), g["prio"]))] = np.arange(n)
        succ = [[] for _ in range(n)]
        for u in range(n):
            for e in range(g["succ_ptr"][u], g["succ_ptr"][u + 1]):
                succ[pi[u]].append(int(pi[g["succ_idx"][e]]))
        ptr = np.zeros(n + 1, np.int64)
        ptr[1:] = np.cumsum([len(s) for s in succ])
        idx = np.array([w for s in succ for w in s], np.int32)
        res2 = np.empty(n, np.int32)
        res2[pi] = g["op_res"]
        prio2 = np.empty(n, np.int32)
        prio2[pi] = rank
        dur2 = np.empty_like(dur)
        dur2[pi] = dur
        mk2, fin2, _ = oracle_run(library, ptr, idx, res2, R, dur2, prio=prio2)
        assert (mk2 == mk).all() and (fin2[pi] == fin).all()


def test_static_replay_of_emergent_order(library):
    """Replaying the oracle's own per-device order reproduces its times."""
    rng = np.random.default_rng(11)
    for _ in range(20):
        n, R = int(rng.integers(1, 40)), int(rng.integers(1, 5))
        g = rand_graph(rng, n, R, 0.1)
        dur = random_durations(n, 1, 1, 50, rng)
        _, fin, _ = run(g, dur, library=library)
        start = fin[:, 0] - dur[:, 0]
        orders = [sorted((v for v in range(n) if g["op_res"][v] == r), key=lambda v: start[v])
                  for r in range(R)]
        ready, f2 = brute._times_for_order(n, preds(g), g["op_res"], dur[:, 0], orders)
        assert f2 == fin[:, 0].tolist()


def test_duplicate_edges_change_nothing(library):
    rng = np.random.default_rng(12)
    for _ in range(20):
        n, R = int(rng.integers(2, 60)), int(rng.integers(1, 5))
        g = rand_graph(rng, n, R, 0.1)
        succ = [list(g["succ_idx"][g["succ_ptr"][u]:g["succ_ptr"][u + 1]]) for u in range(n)]
        for u in range(n):  # repeat some edges, in shuffled positions
            if succ[u] and rng.integers(2):
                succ[u] = list(rng.permutation(succ[u] + list(rng.choice(succ[u], 2))))
        ptr = np.zeros(n + 1, np.int64)
        ptr[1:] = np.cumsum([len(x) for x in succ])
        gd = dict(g, succ_ptr=ptr, succ_idx=np.array([w for x in succ for w in x], np.int32))
        dur = random_durations(n, 3, 1, 20, rng)
        a, b = run(g, dur, library=library), run(gd, dur, library=library)
        assert (a[0] == b[0]).all() and (a[1] == b[1]).all()


def test_placement_overrides_op_res(library):
    """place[v, s] is the resource of v in scenario s (the per-op "device" property)."""
    rng = np.random.default_rng(13)
    n, R, S = 50, 6, 12
    g = rand_graph(rng, n, R, 0.08)
    dur = random_durations(n, S, 1, 30, rng)
    place = rng.integers(0, R, size=(n, S)).astype(np.uint16)
    mk, fin, st = run(g, dur, place=place, library=library)
    assert (st == 0).all()
    for s in range(S):
        gs = dict(g, op_res=place[:, s].astype(np.int32))
        mk1, fin1, _ = run(gs, dur[:, s:s + 1], library=library)
        assert mk1[0] == mk[s] and (fin1[:, 0] == fin[:, s]).all()


# ------------------------------------------------------------ critical path

def test_critical_path_brute_force_and_path(library):
    rng = np.random.default_rng(14)
    for _ in range(60):
        n = int(rng.integers(1, 10))
        g = rand_graph(rng, n, 1, float(rng.uniform(0, 0.6)), dup=bool(rng.integers(2)))
        dur = random_durations(n, 3, 1, 5, rng)
        cp, _ = oracle_cp(library, g["succ_ptr"], g["succ_idx"], n, dur)
        for s in range(3):
            assert cp[s] == brute.all_path_lengths(n, g["succ_ptr"], g["succ_idx"], dur[:, s])
            _, path = oracle_cp(library, g["succ_ptr"], g["succ_idx"], n, dur, s)
            assert dur[path, s].sum() == cp[s]
            P = preds(g)
            assert not P[path[0]]
            for a, b in zip(path, path[1:]):
                assert a in P[b]
            # tie rules: the last op is the lowest id reaching cp; each step back
            # takes the lowest-id predecessor that lies on a longest path
            dist = longest_path_scipy(g, dur[:, s])
            assert path[-1] == int(np.nonzero(dist == cp[s])[0][0])
            for a, b in zip(path, path[1:]):
                cands = [p for p in P[b] if dist[p] == dist[b] - dur[b, s]]
                assert a == min(cands)


# ------------------------------------------------------------------- errors

def test_errors_and_status(library):
    ptr = np.array([0, 1, 1], np.int64)
    idx = np.array([1], np.int32)
    res = np.array([0, 0], np.int32)
    dur = np.array([[1, 0, 5, 1_500_000_000], [1, 1, 5, 1_500_000_000]], np.int32)
    mk, fin, st = oracle_run(library, ptr, idx, res, 1, dur)
    assert st.tolist() == [0, oracle.ST_BAD_DUR, 0, oracle.ST_OVERFLOW]
    assert mk.tolist() == [2, -1, 10, -1]
    cp, _ = oracle_cp(library, ptr, idx, 2, dur)
    assert cp.tolist() == [2, -1, 10, -1]
    place = np.array([[0, 0, 0, 0], [0, 1, 7, 0]], np.uint16)
    mk, _, st = oracle_run(library, ptr, idx, res, 2, dur, place=place)
    assert st.tolist() == [0, oracle.ST_BAD_DUR, oracle.ST_BAD_RES, oracle.ST_OVERFLOW]
    assert mk.tolist() == [2, -1, -1, -1]
    d1 = dur[:, :1]
    with pytest.raises(oracle.OracleError) as e:  # cycle 0 -> 1 -> 0
        oracle_run(library, np.array([0, 1, 2]), np.array([1, 0]), res, 1, d1)
    assert e.value.code == oracle.E_CYCLE
    with pytest.raises(oracle.OracleError) as e:  # self loop
        oracle_run(library, np.array([0, 1, 1]), np.array([0]), res, 1, d1)
    assert e.value.code == oracle.E_CYCLE
    with pytest.raises(oracle.OracleError) as e:  # successor out of range
        oracle_run(library, ptr, np.array([2]), res, 1, d1)
    assert e.value.code == oracle.E_RANGE
    with pytest.raises(oracle.OracleError) as e:  # resource out of range
        oracle_run(library, ptr, idx, np.array([0, 1], np.int32), 1, d1)
    assert e.value.code == oracle.E_RANGE
    with pytest.raises(oracle.OracleError) as e:  # decreasing pointers
        oracle_run(library, np.array([0, 1, 0]), idx, res, 1, d1)
    assert e.value.code == oracle.E_INVAL
    with pytest.raises(oracle.OracleError) as e:
        oracle_cp(library, np.array([0, 1, 2]), np.array([1, 0]), 2, d1)
    assert e.value.code == oracle.E_CYCLE


def test_empty_graph_and_zero_scenarios(library):
    e = np.zeros(1, np.int64)
    mk, fin, st = oracle_run(library, e, np.zeros(0, np.int32), np.zeros(0, np.int32), 1,
                                   np.zeros((0, 5), np.int32))
    assert mk.tolist() == [0] * 5 and st.tolist() == [0] * 5
    cp, _ = oracle_cp(library, e, np.zeros(0, np.int32), 0, np.zeros((0, 5), np.int32))
    assert cp.tolist() == [0] * 5
    mk, _, _ = oracle_run(library, np.array([0, 0]), np.zeros(0, np.int32), np.array([0], np.int32), 1,
                                np.zeros((1, 0), np.int32))
    assert mk.size == 0


def test_threads_do_not_change_results(library):
    rng = np.random.default_rng(15)
    g = rand_graph(rng, 120, 5, 0.04, prio=True)
    dur = random_durations(120, 97, 1, 500, rng)
    a = run(g, dur, n_threads=1, library=library)
    b = run(g, dur, n_threads=7, library=library)
    assert all((x == y).all() for x, y in zip(a, b))


# ------------------------------------------------------ static-order replay

def oracle_static(library, g, order, dur, **kw):
    return oracle.static_run(g["succ_ptr"], g["succ_idx"], g["op_res"], g["n_res"], order, dur,
                             library=library, **kw)


def des_order(g, dur_col, fin_col):
    """All ops sorted by their start time in a replay (ties by op id): on each
    device the starts are strictly increasing, so each device's part of this
    order is the device's own run order."""
    start = fin_col.astype(np.int64) - dur_col
    return np.array(sorted(range(g["n"]), key=lambda v: (start[v], v)), np.int32)


def test_static_single_device_prefix_sums(library):
    """One device, no edges: the ops run back to back in the given order, so
    the finish times are the prefix sums of the durations in that order."""
    rng = np.random.default_rng(21)
    for _ in range(20):
        n = int(rng.integers(1, 50))
        g = dict(n=n, n_res=1, succ_ptr=np.zeros(n + 1, np.int64), succ_idx=np.zeros(0, np.int32),
                 op_res=np.zeros(n, np.int32))
        order = rng.permutation(n).astype(np.int32)
        dur = random_durations(n, 4, 1, 1000, rng)
        mk, fin, st = oracle_static(library, g, order, dur)
        assert (st == 0).all()
        for s in range(4):
            expect = np.cumsum(dur[order, s].astype(np.int64))
            assert (fin[order, s] == expect).all()
            assert mk[s] == expect[-1]


def test_static_own_devices_is_longest_path(library):
    """Every op on its own device: no device order constrains anything and
    the finish times are the longest paths (scipy Bellman-Ford)."""
    rng = np.random.default_rng(22)
    for _ in range(20):
        n = int(rng.integers(1, 60))
        g = rand_graph(rng, n, 1, float(rng.uniform(0, 0.25)), dup=bool(rng.integers(2)))
        g["n_res"], g["op_res"] = n, np.arange(n, dtype=np.int32)
        order = rng.permutation(n).astype(np.int32)
        dur = random_durations(n, 3, 1, 1000, rng)
        mk, fin, _ = oracle_static(library, g, order, dur)
        for s in range(3):
            dist = longest_path_scipy(g, dur[:, s])
            assert (fin[:, s] == dist).all()
            assert mk[s] == dist.max()


def test_static_replays_the_event_order(library):
    """Given the run order that the event replay produced on every device
    (its start order), the static-order replay reproduces that scenario's
    finish times exactly; with several scenarios sharing one order, the
    scenario the order came from is reproduced."""
    rng = np.random.default_rng(23)
    for _ in range(40):
        n, R = int(rng.integers(1, 60)), int(rng.integers(1, 6))
        g = rand_graph(rng, n, R, float(rng.uniform(0, 0.3)), prio=bool(rng.integers(2)),
                       dup=bool(rng.integers(2)))
        dur = random_durations(n, 3, 1, int(rng.choice([3, 50, 10000])), rng)
        _, fin, _ = run(g, dur, library=library)
        for s in range(3):
            order = des_order(g, dur[:, s], fin[:, s])
            mk2, fin2, st2 = oracle_static(library, g, order, dur)
            assert st2[s] == 0
            assert (fin2[:, s] == fin[:, s]).all()
            assert mk2[s] == fin[:, s].max()


def test_static_order_is_respected(library):
    """Structure of every static replay: inputs are ready at the start, each
    device runs its ops in the given order without overlap, and an op starts
    exactly when the later of its inputs and its device's previous op allow."""
    rng = np.random.default_rng(24)
    for _ in range(30):
        n, R = int(rng.integers(1, 40)), int(rng.integers(1, 5))
        g = rand_graph(rng, n, R, float(rng.uniform(0, 0.3)))
        # a topological order of the DAG keeps every device order consistent
        P0 = preds(g)
        topo, done = [], set()
        while len(topo) < n:  # smallest id whose predecessors are all placed
            v = min(v for v in range(n) if v not in done and all(u in done for u in P0[v]))
            topo.append(v)
            done.add(v)
        topo = np.array(topo, np.int32)
        dur = random_durations(n, 2, 1, 100, rng)
        mk, fin, st = oracle_static(library, g, topo, dur)
        assert (st == 0).all()
        P = preds(g)
        for s in range(2):
            f = fin[:, s].astype(np.int64)
            start = f - dur[:, s]
            prev = {}
            for v in topo:
                r = g["op_res"][v]
                ready = max([f[u] for u in P[v]], default=0)
                assert start[v] == max(ready, f[prev[r]] if r in prev else 0)
                prev[r] = v
            assert mk[s] == f.max()


def test_static_errors_and_status(library):
    # order must be a permutation
    g = dict(n=3, n_res=1, succ_ptr=np.array([0, 1, 1, 1], np.int64), succ_idx=np.array([1], np.int32),
             op_res=np.zeros(3, np.int32))
    dur = np.ones((3, 2), np.int32)
    for bad in ([0, 0, 1], [0, 1, 3], [0, 1, -1]):
        with pytest.raises(oracle.OracleError) as e:
            oracle_static(library, g, np.array(bad, np.int32), dur)
        assert e.value.code == oracle.E_INVAL
    # the device order contradicts an edge on the same device
    with pytest.raises(oracle.OracleError) as e:
        oracle_static(library, g, np.array([1, 0, 2], np.int32), dur)
    assert e.value.code == oracle.E_CYCLE
    # a cycle through two devices: a->d and b->c are edges; device 0 runs c
    # before a, device 1 runs d before b
    g2 = dict(n=4, n_res=2, succ_ptr=np.array([0, 1, 2, 2, 2], np.int64), succ_idx=np.array([3, 2], np.int32),
              op_res=np.array([0, 1, 0, 1], np.int32))
    with pytest.raises(oracle.OracleError) as e:
        oracle_static(library, g2, np.array([2, 0, 3, 1], np.int32), np.ones((4, 1), np.int32))
    assert e.value.code == oracle.E_CYCLE
    mk, _, _ = oracle_static(library, g2, np.array([0, 2, 1, 3], np.int32), np.ones((4, 1), np.int32))
    assert mk[0] == 2
    # bad durations and overflow
    dur = np.array([[1, 0, 5, 1_500_000_000],
                    [1, 1, 5, 1_500_000_000],
                    [1, 1, -3, 1]], np.int32)
    mk, _, st = oracle_static(library, g, np.array([0, 1, 2], np.int32), dur)
    assert st.tolist() == [0, oracle.ST_BAD_DUR, oracle.ST_BAD_DUR, oracle.ST_OVERFLOW]
    assert mk.tolist() == [3, -1, -1, -1]


# -------------------------------------------------- bottleneck attribution

def oracle_attr(library, g, dur, place=None, path_scen=-1):
    return oracle.attribute(g["succ_ptr"], g["succ_idx"], g["op_res"], g["n_res"], dur,
                            prio=g.get("prio"), place=place, path_scen=path_scen, library=library)


def test_attribution_hand_examples(library):
    """Two schedules worked by hand.  (1) a (device 0, 3 ns) and b (device 0,
    2 ns) are sources, c (device 1, 4 ns) needs b: a 0-3, b 3-5, c 5-9.  The
    chain from c steps to b (its input, finished at 5), then to a (device 0
    finished a at 3, when b started), which starts at 0: device 0 holds 5 ns
    of the 9, device 1 4 ns.  (2) a (device 0, 3 ns), c (device 1, 1 ns) and
    d (device 1, 2 ns, needs a): d runs 3-5 after device 1 idled from 1 to 3;
    the chain is a, d (3 + 2 ns) and device 1 is busy 3 ns of which the chain
    holds 2."""
    g = dict(n=3, n_res=2, succ_ptr=np.array([0, 0, 1, 1], np.int64), succ_idx=np.array([2], np.int32),
             op_res=np.array([0, 0, 1], np.int32), prio=None)
    mk, st, busy, chain, cops, path = oracle_attr(library, g, np.array([[3], [2], [4]], np.int32), path_scen=0)
    assert mk[0] == 9 and st[0] == 0
    assert chain[:, 0].tolist() == [5, 4] and busy[:, 0].tolist() == [5, 4]
    assert cops[0] == 3 and path.tolist() == [0, 1, 2]
    g = dict(n=3, n_res=2, succ_ptr=np.array([0, 1, 1, 1], np.int64), succ_idx=np.array([2], np.int32),
             op_res=np.array([0, 1, 1], np.int32), prio=None)
    mk, st, busy, chain, cops, path = oracle_attr(library, g, np.array([[3], [1], [2]], np.int32), path_scen=0)
    assert mk[0] == 5
    assert chain[:, 0].tolist() == [3, 2] and busy[:, 0].tolist() == [3, 3]
    assert cops[0] == 2 and path.tolist() == [0, 2]


def test_attribution_chain_covers_makespan(library):
    """The chain has no gaps: per scenario its per-device times sum to the
    makespan; busy time is each device's total duration (a plain sum); the
    chain's share of a device never exceeds its busy time, which never
    exceeds the makespan; the makespan equals the replay's."""
    rng = np.random.default_rng(31)
    for _ in range(40):
        n, R = int(rng.integers(1, 60)), int(rng.integers(1, 6))
        g = rand_graph(rng, n, R, float(rng.uniform(0, 0.3)), prio=bool(rng.integers(2)),
                       dup=bool(rng.integers(2)))
        S = 4
        dur = random_durations(n, S, 1, int(rng.choice([3, 100, 10000])), rng)
        place = rng.integers(0, R, size=(n, S)).astype(np.uint16) if rng.integers(2) else None
        mk, st, busy, chain, cops, _ = oracle_attr(library, g, dur, place=place)
        rmk, _, _ = run(g, dur, library=library, place=place)
        assert (mk == rmk).all() and (st == 0).all()
        res = place.astype(np.int64) if place is not None else np.repeat(g["op_res"][:, None], S, 1)
        for s in range(S):
            expect = np.bincount(res[:, s], weights=dur[:, s], minlength=R).astype(np.int64)
            assert (busy[:, s] == expect).all()
        assert (chain.sum(0) == mk).all()
        assert (chain <= busy).all() and (busy <= mk[None, :]).all()
        assert ((1 <= cops) & (cops <= n)).all()


def test_attribution_own_devices_is_critical_path(library):
    """One device per op: nothing waits for a device, so the chain is the
    critical path (same end and tie rules) and each op on it contributes its
    duration on its own device."""
    rng = np.random.default_rng(32)
    for _ in range(25):
        n = int(rng.integers(1, 50))
        g = rand_graph(rng, n, 1, float(rng.uniform(0, 0.3)), dup=bool(rng.integers(2)))
        g["n_res"], g["op_res"] = n, np.arange(n, dtype=np.int32)
        dur = random_durations(n, 3, 1, int(rng.choice([3, 1000])), rng)
        for s in range(3):
            mk, _, _, chain, cops, path = oracle_attr(library, g, dur, path_scen=s)
            cp, cpath = oracle_cp(library, g["succ_ptr"], g["succ_idx"], n, dur, path_scen=s)
            assert mk[s] == cp[s]
            assert path.tolist() == cpath.tolist() and cops[s] == len(cpath)
            expect = np.zeros(n, np.int64)
            expect[cpath] = dur[cpath, s]
            assert (chain[:, s] == expect).all()


def test_attribution_single_device_chain_is_everything(library):
    """One device never idles while ops remain, so the chain holds every op."""
    rng = np.random.default_rng(33)
    for _ in range(20):
        n = int(rng.integers(1, 50))
        g = rand_graph(rng, n, 1, float(rng.uniform(0, 0.3)), prio=True)
        dur = random_durations(n, 3, 1, 50, rng)
        mk, _, busy, chain, cops, _ = oracle_attr(library, g, dur)
        assert (cops == n).all() and (chain[0] == mk).all() and (busy[0] == mk).all()


def test_attribution_chain_binds(library):
    """Each step of the chain, checked against the replay's finish times: the
    chain ends at the lowest-id op of largest finish and starts at 0; each op
    finishes exactly when the next one starts; a step goes to the lowest-id
    predecessor finishing then if one does, otherwise to the op that ran
    right before on the same device."""
    rng = np.random.default_rng(34)
    for _ in range(60):
        n, R = int(rng.integers(1, 40)), int(rng.integers(1, 5))
        g = rand_graph(rng, n, R, float(rng.uniform(0, 0.4)), prio=bool(rng.integers(2)))
        dur = random_durations(n, 2, 1, int(rng.choice([2, 4, 100])), rng)
        _, fin, _ = run(g, dur, library=library)
        P = preds(g)
        for s in range(2):
            _, _, _, _, cops, path = oracle_attr(library, g, dur, path_scen=s)
            f = fin[:, s].astype(np.int64)
            start = f - dur[:, s]
            assert path[-1] == int(np.flatnonzero(f == f.max())[0])
            assert start[path[0]] == 0 and cops[s] == len(path)
            for u, v in zip(path[:-1], path[1:]):
                assert f[u] == start[v]
                data = [p for p in P[v] if f[p] == start[v]]
                if data:
                    assert u == min(data)
                else:
                    r = g["op_res"][v]
                    assert g["op_res"][u] == r
                    between = [x for x in range(n) if g["op_res"][x] == r and start[u] < start[x] < start[v]]
                    assert not between


def test_attribution_status(library):
    g = dict(n=3, n_res=1, succ_ptr=np.array([0, 1, 2, 2], np.int64), succ_idx=np.array([1, 2], np.int32),
             op_res=np.zeros(3, np.int32), prio=None)
    dur = np.array([[1, 0, 1_500_000_000], [1, 1, 1_500_000_000], [1, 1, 1]], np.int32)
    mk, st, busy, chain, cops, path = oracle_attr(library, g, dur, path_scen=1)
    assert st.tolist() == [0, oracle.ST_BAD_DUR, oracle.ST_OVERFLOW]
    assert mk.tolist() == [3, -1, -1] and cops.tolist() == [3, -1, -1]
    assert busy[:, 1:].tolist() == [[0, 0]] and chain[:, 1:].tolist() == [[0, 0]]
    assert path.tolist() == []


# ------------------------------------------------- scenario generation pins
#
# The generator (oracle.h, oracle_generate) is knob grid x counter-based
# noise.  Its building block, Philox4x32-10, is pinned by the published
# known-answer vectors; the round structure it shares with Philox4x64-10 is
# pinned against numpy's Philox (a 4x64-10 implementation); the integer
# composition is checked against arbitrary-precision arithmetic, and the
# noise's distribution against the moments of an 8-term Irwin-Hall sum.

SIGMA_UNIT = 2.0 * np.sqrt(2.0 * (65536.0**2 - 1.0) / 3.0) / 2.0**40  # relative std per unit of noise


def _kat():
    rows = []
    for line in open(os.path.join(goldens.GOLDEN_DIR, "philox4x32_10.kat")):
        line = line.split("#", 1)[0].split()
        if line:
            rows.append([int(x, 16) for x in line])
    return rows


def test_philox4x32_known_answers(library=None):
    for row in _kat():
        out = oracle.philox4x32_10(row[0:4], row[4:6], library=library)
        assert [int(x) for x in out] == row[6:10]


def test_philox4x64_matches_numpy(library=None):
    rng = np.random.default_rng(11)
    for _ in range(20):
        ctr = rng.integers(1, 2**63, size=4, dtype=np.uint64)
        key = rng.integers(0, 2**63, size=2, dtype=np.uint64)
        before = ctr.copy()
        before[0] -= np.uint64(1)  # numpy advances the counter before each block
        ref = np.random.Philox(counter=before, key=key).random_raw(4)
        assert np.array_equal(oracle.philox4x64_10(ctr, key, library=library), ref)


def _gen_exact(base_row_of, S, v, noise, seed, library=None):
    """One generated duration with Python integers, from the pinned Philox block."""
    b = base_row_of(S)[v]
    if b < 1 or b > 2**24:
        return 0
    x = oracle.philox4x32_10([S & 0xFFFFFFFF, S >> 32, v, 0], [seed & 0xFFFFFFFF, seed >> 32],
                             library=library)
    U = sum(int(w) & 0xFFFF for w in x) + sum(int(w) >> 16 for w in x)
    t = 2 * U - 524280
    return b + ((b * t * noise + 2**39) >> 40)


def test_generate_exact_integer_composition(library=None):
    rng = np.random.default_rng(5)
    n, K, kb = 7, 3, 5
    base = rng.integers(1, 2**24, size=(K, n), endpoint=True).astype(np.int32)
    base[0, 0], base[1, 1], base[2, 2] = 1, 2**24, 2**24  # extremes of the valid range
    base[0, 3] = 0  # invalid bases give 0
    base[1, 4] = 2**24 + 1
    for noise in (0, 1, 102739, 2**20 - 1):
        for seed in (0, 2**64 - 1, 0x123456789ABCDEF):
            scen0 = 2**32 - 6  # the counter's high word changes inside the batch
            S_n = 12
            got = oracle.generate(base, S_n, kb, noise, seed, scen0=scen0, library=library)
            for s in range(S_n):
                S = scen0 + s
                for v in range(n):
                    want = _gen_exact(lambda S: base[(S // kb) % K].tolist(), S, v, noise, seed, library)
                    assert got[v, s] == want, (noise, seed, s, v)


def test_generate_knob_grid_without_noise(library=None):
    n, K, kb = 5, 4, 3
    base = np.array([[1000 * (k + 1) + v for v in range(n)] for k in range(K)], np.int32)
    dur = oracle.generate(base, 40, kb, 0, 99, scen0=7, library=library)
    for s in range(40):
        k = ((7 + s) // kb) % K
        assert np.array_equal(dur[:, s], base[k])


def test_generate_global_scenario_index(library=None):
    base = np.arange(1, 9, dtype=np.int32)[None, :] * 10_000
    full = oracle.generate(base, 300, 16, 102739, 42, library=library)
    part = oracle.generate(base, 100, 16, 102739, 42, scen0=150, library=library)
    assert np.array_equal(part, full[:, 150:250])
    other = oracle.generate(base, 300, 16, 102739, 43, library=library)
    assert not np.array_equal(other, full)


def test_generate_noise_moments(library=None):
    b, noise = 1_000_000, 102739  # relative sigma 0.01
    base = np.full((1, 50), b, np.int32)
    dur = oracle.generate(base, 4000, 1, noise, 2024, library=library).astype(np.float64)
    r = dur / b - 1.0
    sigma = noise * SIGMA_UNIT
    assert abs(sigma - 0.01) < 1e-6
    N = r.size
    assert abs(r.mean()) < 4 * sigma / np.sqrt(N)
    assert abs(r.std() / sigma - 1.0) < 0.01
    z = (r - r.mean()) / r.std()
    assert abs((z**3).mean()) < 0.03
    # excess kurtosis of a sum of 8 uniforms is -6/(5*8) = -0.15
    assert abs((z**4).mean() - 3.0 + 0.15) < 0.04
    lim = b * 524280 * noise / 2**40 + 1
    assert np.abs(dur - b).max() <= lim
    # neighbouring counters are uncorrelated
    assert abs(np.corrcoef(r[:, :-1].ravel(), r[:, 1:].ravel())[0, 1]) < 0.02
    assert abs(np.corrcoef(r[:-1].ravel(), r[1:].ravel())[0, 1]) < 0.02


def test_generate_invalid_base_flags_scenario(library=None):
    g = dict(n=3, n_res=1, succ_ptr=np.array([0, 1, 2, 2], np.int64),
             succ_idx=np.array([1, 2], np.int32), op_res=np.zeros(3, np.int32), prio=None)
    base = np.array([[10, 0, 10], [10, 20, 10]], np.int32)
    dur = oracle.generate(base, 4, 1, 0, 0, library=library)
    mk, _, st = run(g, dur, library=library)
    assert list(st) == [ORC_BAD, 0, ORC_BAD, 0]
    assert list(mk) == [-1, 40, -1, 40]


ORC_BAD = oracle.ST_BAD_DUR


def test_generate_argument_errors(library=None):
    base = np.ones((1, 3), np.int32)
    for kw in (dict(knob_block=0), dict(noise=2**20), dict(scen0=-1)):
        args = dict(knob_block=1, noise=0, seed=0, scen0=0)
        args.update(kw)
        with pytest.raises(oracle.OracleError):
            oracle.generate(base, 4, args["knob_block"], args["noise"], args["seed"],
                            scen0=args["scen0"], library=library)


# ------------------------------------------------------ device gap pins
#
# oracle_run_batch_gap: after a device finishes an op it idles gap[r] ns
# before its next op (the paper names this gap as unmodelled, Sec. 3).

def run_gap(g, dur, gap, library=None, **kw):
    return oracle.run_batch(g["succ_ptr"], g["succ_idx"], g["op_res"], g["n_res"], dur,
                            prio=g.get("prio"), library=library, gap=np.asarray(gap, np.int32), **kw)


def test_gap_hand_example(library=None):
    # R0 has a 3 ns gap, R1 none.  op0 (R0, 5), op1 (R1, 2), op2 (R0, 4, after
    # op1), op3 (R0, 1).  t=0: R0 runs op0 [0,5), R1 runs op1 [0,2); t=2: op2
    # ready; R0 is free again at 5+3=8 and serves op3 (ready 0) [8,9), then is
    # free at 12 and serves op2 (ready 2) [12,16).  Without the gap: [5,2,10,6].
    g = dict(n=4, n_res=2, succ_ptr=np.array([0, 0, 1, 1, 1], np.int64), succ_idx=np.array([2], np.int32),
             op_res=np.array([0, 1, 0, 0], np.int32), prio=None)
    dur = np.array([[5], [2], [4], [1]], np.int32)
    mk, fin, st = run_gap(g, dur, [3, 0], library)
    assert list(fin[:, 0]) == [5, 2, 16, 9] and mk[0] == 16 and st[0] == 0
    mk0, fin0, _ = run_gap(g, dur, [0, 0], library)
    assert list(fin0[:, 0]) == [5, 2, 10, 6] and mk0[0] == 10


def test_gap_one_device_closed_form(library=None):
    rng = np.random.default_rng(21)
    n = 9
    g = dict(n=n, n_res=1, succ_ptr=np.zeros(n + 1, np.int64), succ_idx=np.zeros(0, np.int32),
             op_res=np.zeros(n, np.int32), prio=rng.permutation(n).astype(np.int32))
    dur = rng.integers(1, 50, size=(n, 6)).astype(np.int32)
    gap = 7
    mk, fin, _ = run_gap(g, dur, [gap], library)
    order = np.argsort(g["prio"], kind="stable")
    for s in range(dur.shape[1]):
        f = np.cumsum(dur[order, s]) + gap * np.arange(n)
        assert np.array_equal(fin[order, s], f)
        assert mk[s] == dur[:, s].sum() + gap * (n - 1)


def test_gap_chain_closed_forms(library=None):
    rng = np.random.default_rng(22)
    n = 10
    ptr = np.r_[np.arange(n, dtype=np.int64), n - 1]
    idx = np.arange(1, n, dtype=np.int32)
    dur = rng.integers(1, 30, size=(n, 5)).astype(np.int32)
    # one device: every op waits its predecessor's finish plus the gap
    g1 = dict(n=n, n_res=1, succ_ptr=ptr, succ_idx=idx, op_res=np.zeros(n, np.int32), prio=None)
    _, fin, _ = run_gap(g1, dur, [4], library)
    assert np.array_equal(fin, np.cumsum(dur, axis=0) + 4 * np.arange(n)[:, None])
    # two alternating devices: op k's device last ran op k-2, so op k starts
    # at max(f(k-1), f(k-2) + gap)
    g2 = dict(n=n, n_res=2, succ_ptr=ptr, succ_idx=idx, op_res=(np.arange(n) % 2).astype(np.int32), prio=None)
    gap = 12
    _, fin, _ = run_gap(g2, dur, [gap, gap], library)
    for s in range(dur.shape[1]):
        f = [int(dur[0, s]), int(dur[0, s] + dur[1, s])]
        for k in range(2, n):
            f.append(max(f[-1], f[-2] + gap) + int(dur[k, s]))
        assert list(fin[:, s]) == f


def test_gap_one_device_per_op_is_longest_path(library=None):
    rng = np.random.default_rng(23)
    for _ in range(5):
        n = 14
        g = rand_graph(rng, n, n, 0.25)
        g["op_res"] = np.arange(n, dtype=np.int32)
        dur = rng.integers(1, 100, size=(n, 4)).astype(np.int32)
        mk, fin, _ = run_gap(g, dur, rng.integers(0, 1000, size=n), library)
        mk0, fin0, _ = run(g, dur, library=library)
        assert np.array_equal(fin, fin0) and np.array_equal(mk, mk0)


def test_gap_matches_brute_force(library=None):
    rng = np.random.default_rng(24)
    for trial in range(40):
        n = int(rng.integers(2, 7))
        R = int(rng.integers(1, 3))
        g = rand_graph(rng, n, R, 0.35, prio=trial % 2 == 0)
        dur = rng.integers(1, 6, size=(n, 1)).astype(np.int32)
        gap = rng.integers(0, 5, size=R).astype(np.int32)
        mk, fin, st = run_gap(g, dur, gap, library)
        assert st[0] == 0
        tick = brute.tick_sim(n, R, g["succ_ptr"], g["succ_idx"], g["op_res"], dur[:, 0], g["prio"], gap=gap)
        assert list(fin[:, 0]) == tick
        found = brute.enumerate_orders(n, R, g["succ_ptr"], g["succ_idx"], g["op_res"], dur[:, 0], g["prio"],
                                       gap=gap)
        assert found == [tick]


def test_gap_bounds(library=None):
    rng = np.random.default_rng(25)
    for _ in range(6):
        n, R = 40, 4
        g = rand_graph(rng, n, R, 0.08)
        dur = rng.integers(1, 200, size=(n, 8)).astype(np.int32)
        gap = rng.integers(0, 150, size=R).astype(np.int32)
        mk, fin, _ = run_gap(g, dur, gap, library)
        cp, _ = oracle.critical_path(g["succ_ptr"], g["succ_idx"], n, dur, library=library)
        cnt = np.bincount(g["op_res"], minlength=R)
        for s in range(dur.shape[1]):
            busy = np.bincount(g["op_res"], weights=dur[:, s], minlength=R)
            lower = max(cp[s], int((busy + gap * np.maximum(cnt - 1, 0)).max()))
            upper = int(dur[:, s].sum() + (gap * np.maximum(cnt - 1, 0)).sum())
            assert lower <= mk[s] <= upper
            # consecutive ops on a device are at least the gap apart
            start = fin[:, s] - dur[:, s]
            for r in range(R):
                ops = np.nonzero(g["op_res"] == r)[0]
                o = ops[np.argsort(start[ops])]
                assert (start[o[1:]] >= fin[o[:-1], s] + gap[r]).all()


def test_gap_errors_and_overflow(library=None):
    g = dict(n=2, n_res=1, succ_ptr=np.array([0, 0, 0], np.int64), succ_idx=np.zeros(0, np.int32),
             op_res=np.zeros(2, np.int32), prio=None)
    with pytest.raises(oracle.OracleError):
        run_gap(g, np.ones((2, 1), np.int32), [-1], library)
    # two ops of 2^30 ns with a 2^30 - 1 ns gap between them pass INT32_MAX;
    # 2^29 and 1 ns with that gap end at 2^29 + 2^30
    dur = np.array([[2**30, 2**29], [2**30, 1]], np.int32)
    mk, _, st = run_gap(g, dur, [2**30 - 1], library)
    assert st[0] == oracle.ST_OVERFLOW and mk[0] == -1
    assert st[1] == 0 and mk[1] == 2**29 + 2**30


# ----------------------------------------------------- output delay pins
#
# oracle_run_batch_dev: an op on device r hands its outputs to its
# successors delay[r] ns after it finishes (the memcpy time the paper lists
# as unmodelled, Sec. 3); the device itself is free at the finish (plus gap).

def run_dev(g, dur, gap=None, delay=None, library=None, **kw):
    return oracle.run_batch(g["succ_ptr"], g["succ_idx"], g["op_res"], g["n_res"], dur, prio=g.get("prio"),
                            library=library, gap=None if gap is None else np.asarray(gap, np.int32),
                            delay=np.asarray(delay, np.int32), **kw)


def test_delay_hand_example(library=None):
    # op0 (R0, 5) -> op1 (R1, 3); op2 (R0, 2).  R0's outputs take 4 ns to
    # arrive: op1 is ready at 9 and ends at 12, while R0 is free at 5 and
    # runs op2 over [5, 7).  Without the delay op1 ends at 8.
    g = dict(n=3, n_res=2, succ_ptr=np.array([0, 1, 1, 1], np.int64), succ_idx=np.array([1], np.int32),
             op_res=np.array([0, 1, 0], np.int32), prio=None)
    dur = np.array([[5], [3], [2]], np.int32)
    mk, fin, st = run_dev(g, dur, delay=[4, 0], library=library)
    assert list(fin[:, 0]) == [5, 12, 7] and mk[0] == 12 and st[0] == 0
    mk, fin, _ = run_dev(g, dur, delay=[0, 100], library=library)  # R1's delay: no successors
    assert list(fin[:, 0]) == [5, 8, 7] and mk[0] == 8


def test_delay_one_device_per_op_is_weighted_longest_path(library=None):
    rng = np.random.default_rng(31)
    for _ in range(5):
        n = 15
        g = rand_graph(rng, n, n, 0.25)
        g["op_res"] = np.arange(n, dtype=np.int32)
        dur = rng.integers(1, 100, size=(n, 3)).astype(np.int32)
        delay = rng.integers(0, 50, size=n).astype(np.int32)
        mk, fin, _ = run_dev(g, dur, delay=delay, library=library)
        for s in range(3):
            # longest path from a super-source: node n -> v weighs d(v),
            # u -> v weighs delay(u) + d(v); scipy finds it on negated weights
            rows, cols, wts = [], [], []
            for v in range(n):
                rows.append(n), cols.append(v), wts.append(-float(dur[v, s]))
            for u in range(n):
                for e in range(g["succ_ptr"][u], g["succ_ptr"][u + 1]):
                    v = int(g["succ_idx"][e])
                    rows.append(u), cols.append(v), wts.append(-float(delay[u] + dur[v, s]))
            A = scipy.sparse.csr_matrix((wts, (rows, cols)), shape=(n + 1, n + 1))
            dist = scipy.sparse.csgraph.bellman_ford(A, indices=n)
            assert np.array_equal(fin[:, s], (-dist[:n]).astype(np.int64))


def test_delay_chain_closed_form(library=None):
    rng = np.random.default_rng(32)
    n = 10
    ptr = np.r_[np.arange(n, dtype=np.int64), n - 1]
    idx = np.arange(1, n, dtype=np.int32)
    g = dict(n=n, n_res=2, succ_ptr=ptr, succ_idx=idx, op_res=(np.arange(n) % 2).astype(np.int32), prio=None)
    dur = rng.integers(1, 30, size=(n, 4)).astype(np.int32)
    gap, delay = [6, 9], [11, 3]
    _, fin, _ = run_dev(g, dur, gap=gap, delay=delay, library=library)
    for s in range(4):
        f = [int(dur[0, s])]
        for k in range(1, n):  # ready when the previous op's outputs arrive; the device after its gap
            start = f[-1] + delay[(k - 1) % 2]
            if k >= 2:
                start = max(start, f[-2] + gap[k % 2])
            f.append(start + int(dur[k, s]))
        assert list(fin[:, s]) == f


def test_delay_matches_brute_force(library=None):
    rng = np.random.default_rng(33)
    for trial in range(40):
        n = int(rng.integers(2, 7))
        R = int(rng.integers(1, 3))
        g = rand_graph(rng, n, R, 0.4, prio=trial % 2 == 0)
        dur = rng.integers(1, 6, size=(n, 1)).astype(np.int32)
        gap = rng.integers(0, 4, size=R).astype(np.int32)
        delay = rng.integers(0, 5, size=R).astype(np.int32)
        mk, fin, st = run_dev(g, dur, gap=gap, delay=delay, library=library)
        assert st[0] == 0
        tick = brute.tick_sim(n, R, g["succ_ptr"], g["succ_idx"], g["op_res"], dur[:, 0], g["prio"], gap=gap,
                              delay=delay)
        assert list(fin[:, 0]) == tick
        found = brute.enumerate_orders(n, R, g["succ_ptr"], g["succ_idx"], g["op_res"], dur[:, 0], g["prio"],
                                       gap=gap, delay=delay)
        assert found == [tick]


def test_delay_zero_and_errors(library=None):
    rng = np.random.default_rng(34)
    g = rand_graph(rng, 30, 3, 0.1)
    dur = rng.integers(1, 100, size=(30, 6)).astype(np.int32)
    mk0, fin0, _ = run(g, dur, library=library)
    mk, fin, _ = run_dev(g, dur, delay=[0, 0, 0], library=library)
    assert np.array_equal(mk, mk0) and np.array_equal(fin, fin0)
    with pytest.raises(oracle.OracleError):
        run_dev(g, dur, delay=[0, -1, 0], library=library)


# ---------------------------------------------------------------- bandwidth sharing


def run_share(g, dur, share, library=None, **kw):
    return oracle.run_batch_share(g["succ_ptr"], g["succ_idx"], g["op_res"], g["n_res"], dur, share=share,
                                  prio=g.get("prio"), library=library, **kw)


def no_edges(res):
    n = len(res)
    return dict(n=n, n_res=int(max(res)) + 1, succ_ptr=np.zeros(n + 1, np.int64), succ_idx=np.zeros(0, np.int32),
                op_res=np.asarray(res, np.int32), prio=None)


def test_share_hand_example(library=None):
    # op0 (d 10) on shared link 0 from t = 0; op1 (device 1, 4) -> op2 (link
    # 0, d 2).  Alone over [0, 4) op0 receives 4 ns; from 4 the two share:
    # op2 needs 2 ns of service, which takes 4 ns, so it leaves at 8; op0
    # then holds 6 and finishes its last 4 ns alone at 12.
    g = dict(n=3, n_res=2, succ_ptr=np.array([0, 0, 1, 1], np.int64), succ_idx=np.array([2], np.int32),
             op_res=np.array([0, 1, 0], np.int32), prio=None)
    dur = np.array([[10], [4], [2]], np.int32)
    mk, fin, st = run_share(g, dur, [1, 0], library=library)
    assert list(fin[:, 0]) == [12, 4, 8] and mk[0] == 12 and st[0] == 0
    mk, fin, _ = run_share(g, dur, [0, 0], library=library)  # exclusive: op2 waits for op0
    assert list(fin[:, 0]) == [10, 4, 12] and mk[0] == 12
    # equal sharing from one start: 4 and 10 -> 8 and 14; three of 3 -> 9
    mk, fin, _ = run_share(no_edges([0, 0]), np.array([[4], [10]], np.int32), [1], library=library)
    assert list(fin[:, 0]) == [8, 14]
    mk, fin, _ = run_share(no_edges([0, 0, 0]), np.full((3, 1), 3, np.int32), [1], library=library)
    assert list(fin[:, 0]) == [9, 9, 9]
    # ties: ops 0 and 1 share link 0 and both leave at 4, when op 2 also ends
    # on device 1.  Op 3 (after op 0) and op 4 (after op 2) become ready on
    # device 2 at 4; the lower id runs first, although op 4 was known to be
    # ready at 4 before the link's finishes at 4 were taken.
    g = dict(n=5, n_res=3, succ_ptr=np.array([0, 1, 1, 2, 2, 2], np.int64), succ_idx=np.array([3, 4], np.int32),
             op_res=np.array([0, 0, 1, 2, 2], np.int32), prio=None)
    dur = np.array([[2], [2], [4], [5], [5]], np.int32)
    _, fin, _ = run_share(g, dur, [1, 0, 0], library=library)
    assert list(fin[:, 0]) == [4, 4, 4, 9, 14]


def test_share_simultaneous_start_closed_form(library=None):
    # k ops entering one shared link together leave in order of duration;
    # the i-th (ascending d) at sum_{j<i} d_j + (k - i) d_i (0-based i)
    assert oracle.SHARE_UNIT == 4096 * math.lcm(*range(1, 17)) < 2**32
    rng = np.random.default_rng(41)
    for k in (1, 2, 5, 16):  # every count 1..k divides the service unit: exact shares
        g = no_edges([0] * k)
        dur = rng.integers(1, 1000, size=(k, 8)).astype(np.int32)
        _, fin, st = run_share(g, dur, [1], library=library)
        assert (st == 0).all()
        for s in range(8):
            d = np.sort(dur[:, s].astype(np.int64))
            want = np.cumsum(np.r_[0, d[:-1]]) + (k - np.arange(k)) * d
            order = np.argsort(dur[:, s], kind="stable")
            assert np.array_equal(np.sort(fin[:, s]), want)
            assert np.all(np.diff(fin[order, s]) >= 0)  # shorter never leaves later
            assert fin[:, s].max() == d.sum()  # the link never idles: work conserved
    # above 16 some counts do not divide the unit: an op gets its share
    # rounded down, and a finish is seen at the next whole ns while the
    # others still share with it, so each op leaves no earlier than under
    # exact sharing and a few ns later at most
    for k in (17, 25, 64):
        g = no_edges([0] * k)
        dur = rng.integers(1, 1000, size=(k, 8)).astype(np.int32)
        _, fin, st = run_share(g, dur, [1], library=library)
        assert (st == 0).all()
        for s in range(8):
            d = np.sort(dur[:, s].astype(np.int64))
            want = np.cumsum(np.r_[0, d[:-1]]) + (k - np.arange(k)) * d
            got = np.sort(fin[:, s])
            assert np.all(got >= want) and np.all(got <= want + k)


def test_share_matches_tick_simulation(library=None):
    rng = np.random.default_rng(42)
    for trial in range(60):
        n = int(rng.integers(2, 12))
        R = int(rng.integers(1, 4))
        g = rand_graph(rng, n, R, 0.3, prio=trial % 2 == 0)
        share = (rng.random(R) < 0.6).astype(np.uint8)
        dur = rng.integers(1, 9, size=(n, 1)).astype(np.int32)
        mk, fin, st = run_share(g, dur, share, library=library)
        assert st[0] == 0
        tick = brute.tick_sim_share(n, R, g["succ_ptr"], g["succ_idx"], g["op_res"], dur[:, 0], share, g["prio"])
        assert list(fin[:, 0]) == tick, (trial, share)
        assert mk[0] == max(tick)


def test_share_worked_examples(library=None):
    """Hand-derived schedules with 17 and 25 ops sharing one link, where the
    count does not divide the service unit (tests/golden/share_*.txt)."""
    for g in goldens.share_goldens():
        ex = g["expect"]
        mk, fin, st = run_share(g, g["dur"], np.array(ex["shared"], np.uint8), library=library)
        assert st.tolist() == [0], g["name"]
        assert fin[:, 0].tolist() == ex["finish"], g["name"]
        assert mk.tolist() == ex["makespan"], g["name"]
        tick = brute.tick_sim_share_units(g["n"], g["n_res"], g["succ_ptr"], g["succ_idx"], g["op_res"],
                                          g["dur"][:, 0], ex["shared"], oracle.SHARE_UNIT, g["prio"])
        assert tick == ex["finish"], g["name"]


def test_share_floor_rule_matches_unit_tick_simulation(library=None):
    """Above 16 active ops the share per ns is the service unit divided by
    the count, rounded down: the oracle equals a 1-ns integer tick simulation
    of that rule exactly, for counts that do not divide the unit (17, 19, 25,
    61), for counts that do (63, 64), and on random graphs whose links reach
    more than 16."""
    U = oracle.SHARE_UNIT
    rng = np.random.default_rng(45)
    for k in (17, 19, 25, 61, 63, 64):
        assert (k >= 63) == (U % k == 0)
        g = no_edges([0] * k)
        dur = rng.integers(1, 12, size=(k, 3)).astype(np.int32)
        _, fin, st = run_share(g, dur, [1], library=library)
        assert (st == 0).all()
        for s in range(3):
            tick = brute.tick_sim_share_units(k, 1, g["succ_ptr"], g["succ_idx"], g["op_res"], dur[:, s], [1], U)
            assert list(fin[:, s]) == tick, (k, s)
        # staggered arrivals: op i becomes ready after a chain of i % 4 exclusive ops
        n = k + 3
        preds = [[] for _ in range(n)]
        for i in range(k):
            if i % 4:
                preds[i].append(k + (i % 4) - 1)
        preds[k + 1].append(k)
        preds[k + 2].append(k + 1)
        succ = [[] for _ in range(n)]
        for v in range(n):
            for u in preds[v]:
                succ[u].append(v)
        gg = dict(n=n, n_res=2, succ_ptr=np.r_[0, np.cumsum([len(x) for x in succ])].astype(np.int64),
                  succ_idx=np.array([w for x in succ for w in x], np.int32),
                  op_res=np.array([0] * k + [1] * 3, np.int32), prio=None)
        dd = rng.integers(1, 9, size=(n, 2)).astype(np.int32)
        _, fin, st = run_share(gg, dd, [1, 0], library=library)
        assert (st == 0).all()
        for s in range(2):
            tick = brute.tick_sim_share_units(n, 2, gg["succ_ptr"], gg["succ_idx"], gg["op_res"], dd[:, s], [1, 0], U)
            assert list(fin[:, s]) == tick, (k, s)
    seen_big = 0
    for trial in range(12):
        n = int(rng.integers(30, 60))
        g = rand_graph(rng, n, 2, 0.02, prio=trial % 2 == 0)
        g["op_res"] = (rng.random(n) < 0.8).astype(np.int32) ^ 1  # about 80 % on shared device 0
        dur = rng.integers(1, 6, size=(n, 1)).astype(np.int32)
        share = np.array([1, 0], np.uint8)
        mk, fin, st = run_share(g, dur, share, library=library)
        assert st[0] == 0
        tick = brute.tick_sim_share_units(n, 2, g["succ_ptr"], g["succ_idx"], g["op_res"], dur[:, 0], share, U,
                                          g["prio"])
        assert list(fin[:, 0]) == tick, trial
        srcs = [v for v in range(n) if g["op_res"][v] == 0 and not any(
            v in g["succ_idx"][g["succ_ptr"][u]:g["succ_ptr"][u + 1]] for u in range(n))]
        seen_big += len(srcs) > 16
    assert seen_big >= 6  # most trials start more than 16 ops at once on the link


def test_share_off_or_without_overlap_is_the_plain_replay(library=None):
    rng = np.random.default_rng(43)
    g = rand_graph(rng, 40, 4, 0.1, prio=True)
    dur = rng.integers(1, 100, size=(40, 5)).astype(np.int32)
    mk0, fin0, _ = run(g, dur, library=library)
    mk, fin, _ = run_share(g, dur, [0, 0, 0, 0], library=library)
    assert np.array_equal(mk, mk0) and np.array_equal(fin, fin0)
    mk, fin, _ = run_share(g, dur, None, library=library)
    assert np.array_equal(fin, fin0)
    # a chain never has two ops at once, so sharing changes nothing
    n = 12
    chain = dict(n=n, n_res=2, succ_ptr=np.r_[np.arange(n, dtype=np.int64), n - 1],
                 succ_idx=np.arange(1, n, dtype=np.int32), op_res=(np.arange(n) % 2).astype(np.int32), prio=None)
    cd = rng.integers(1, 50, size=(n, 3)).astype(np.int32)
    _, f0, _ = run(chain, cd, library=library)
    _, f1, _ = run_share(chain, cd, [1, 1], library=library)
    assert np.array_equal(f0, f1)
    # one op per shared device: never shared, the critical path
    one = rand_graph(rng, 20, 20, 0.2)
    one["op_res"] = np.arange(20, dtype=np.int32)
    od = rng.integers(1, 50, size=(20, 3)).astype(np.int32)
    mk, _, _ = run_share(one, od, np.ones(20, np.uint8), library=library)
    cp, _ = oracle.critical_path(one["succ_ptr"], one["succ_idx"], 20, od, library=library)
    assert np.array_equal(mk, cp)


def test_share_bounds(library=None):
    # with every device shared: critical path <= makespan, and each device
    # is work conserving, so makespan <= sum of durations + one ns per op
    rng = np.random.default_rng(44)
    for _ in range(10):
        g = rand_graph(rng, 30, 3, 0.08)
        dur = rng.integers(1, 200, size=(30, 4)).astype(np.int32)
        mk, fin, st = run_share(g, dur, [1, 1, 1], library=library)
        cp, _ = oracle.critical_path(g["succ_ptr"], g["succ_idx"], 30, dur, library=library)
        assert (st == 0).all() and (mk >= cp).all() and (mk <= dur.sum(0) + 30).all()
        for v in range(30):  # an op takes at least its duration
            for e in range(g["succ_ptr"][v], g["succ_ptr"][v + 1]):
                assert (fin[g["succ_idx"][e]] >= fin[v] + dur[g["succ_idx"][e]]).all()


def test_share_limit_overflow_and_errors(library=None):
    m = oracle.SHARE_MAX
    dur = np.full((m + 1, 2), 5, np.int32)
    dur[3, 1] = 0
    mk, _, st = run_share(no_edges([0] * (m + 1)), dur, [1], library=library)
    assert st[0] == oracle.ST_SHARE_LIMIT and mk[0] == -1 and st[1] == oracle.ST_BAD_DUR
    mk, fin, st = run_share(no_edges([0] * m), dur[:m, :1], [1], library=library)
    assert st[0] == 0 and (fin[:, 0] == 5 * m).all()  # 64 divides the unit: exact shares
    big = np.full((2, 1), 2**30 + 1, np.int32)  # two shared ops of 2^30 + 1: both end at 2^31 + 2
    mk, _, st = run_share(no_edges([0, 0]), big, [1], library=library)
    assert st[0] == oracle.ST_OVERFLOW and mk[0] == -1
    mk, _, st = run_share(no_edges([0, 0]), big, [0], library=library)  # exclusive: also overflows
    assert st[0] == oracle.ST_OVERFLOW
    with pytest.raises(oracle.OracleError):
        oracle.run_batch_share(np.array([0, 1, 1], np.int64), np.array([0], np.int32), np.zeros(2, np.int32), 1,
                               np.ones((2, 1), np.int32), share=[1], library=library)
