"""GPU parity of the replay with a device model (sim_run_batch_dev): a gap
per resource between consecutive ops and an output delay per resource.

The outputs of an op that finishes at f on resource r reach its successors
at f + delay[r]; the resource itself is free at f (or f + gap[r]).  Every
case calls the library through its C ABI and compares the integer outputs
element by element with the oracle's replay with gaps and delays.
"""
import os

import numpy as np
import pytest

import oracle
from paper_2002_06790_amd import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mlsim():
    import paper_2002_06790_amd as m
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    if not os.path.exists(m.LIB_PATH):
        m.build()
    return m


def dev(a, dtype=torch.int32):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dtype=dtype, device="cuda")


def dev_place(place):
    return None if place is None else torch.from_numpy(np.ascontiguousarray(place).view(np.int16)).cuda().view(
        torch.uint16)


def check(mlsim, ptr, idx, res, R, dur, gap, delay, prio=None, place=None):
    g = mlsim.Graph(ptr, idx, res, R, prio=prio)
    mk, fin, st = g.run(dev(dur), place=dev_place(place), want_finish=True, algo="event", gap=gap, delay=delay)
    torch.cuda.synchronize()
    omk, ofin, ost = oracle.run_batch(ptr, idx, res, R, dur, prio=prio, place=place, gap=gap, delay=delay)
    st = st.cpu().numpy()
    assert np.array_equal(st, ost), "status differs"
    assert np.array_equal(mk.cpu().numpy(), omk), "makespan differs"
    ok = ost == 0
    assert np.array_equal(fin.cpu().numpy()[:, ok], ofin[:, ok]), "finish times differ"
    g.close()
    return omk, ost


def test_hand_example(mlsim):
    # op0 (R0, 5) -> op1 (R1, 3); op2 (R0, 2).  R0's outputs arrive 4 ns
    # after op0 ends: op1 runs over [9, 12) while R0 runs op2 over [5, 7).
    ptr = np.array([0, 1, 1, 1], np.int64)
    idx = np.array([1], np.int32)
    res = np.array([0, 1, 0], np.int32)
    dur = np.array([[5], [3], [2]], np.int32)
    g = mlsim.Graph(ptr, idx, res, 2)
    mk, fin, _ = g.run(dev(dur), want_finish=True, delay=[4, 0])
    torch.cuda.synchronize()
    assert fin.cpu().numpy()[:, 0].tolist() == [5, 12, 7] and int(mk[0]) == 12
    mk, fin, _ = g.run(dev(dur), want_finish=True, delay=[0, 100])  # a sink's delay does not count
    torch.cuda.synchronize()
    assert fin.cpu().numpy()[:, 0].tolist() == [5, 8, 7] and int(mk[0]) == 8
    g.close()


@pytest.mark.parametrize("k,S", [(1, 1024), (2, 200), (3, 333), (4, 200), (5, 130)])
def test_workload_parity(mlsim, k, S):
    w = W.make_config(k, n_scen=S if k != 1 else None)
    dur = w.durations()
    rng = np.random.default_rng(100 + k)
    delay = rng.integers(0, 30_000, size=w.n_res).astype(np.int32)
    delay[0] = 0
    gap = rng.integers(0, 5_000, size=w.n_res).astype(np.int32) if k % 2 else None
    print(f"delay workload {w.name} S={dur.shape[1]} gaps={gap is not None}", flush=True)
    check(mlsim, w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur, gap, delay, prio=w.prio, place=w.placement())


def test_zero_delays_equal_plain_and_gap_replay(mlsim):
    w = W.make_config(4, n_scen=256)
    dur = w.durations()
    g = mlsim.Graph.from_workload(w)
    d = dev(dur)
    zero = np.zeros(w.n_res, np.int32)
    gap = np.full(w.n_res, 1_500, np.int32)
    mk, fin, st = g.run(d, want_finish=True, algo="event")
    dmk, dfin, dst = g.run(d, want_finish=True, delay=zero)
    torch.cuda.synchronize()
    assert torch.equal(mk, dmk) and torch.equal(fin, dfin) and torch.equal(st, dst)
    pmk, pfin, pst = g.run(d, want_finish=True, gap=gap)
    qmk, qfin, qst = g.run(d, want_finish=True, gap=gap, delay=zero)
    torch.cuda.synchronize()
    assert torch.equal(pmk, qmk) and torch.equal(pfin, qfin) and torch.equal(pst, qst)
    g.close()


def fan_graph(rng, n_src, width):
    """Sources each releasing a fan of 2..width ops whose only predecessor
    it is, each fan op with no successor or one that has a single
    predecessor (the ops the library may chain), a few fan ops that also
    join two fans (not chained), and one sink joining everything left
    open.  Returns (succ_ptr, succ_idx, n)."""
    succ, n = [], 0

    def new():
        nonlocal n
        succ.append([])
        n += 1
        return n - 1

    srcs = [new() for _ in range(n_src)]
    fans = []
    for u in srcs:
        fan = [new() for _ in range(int(rng.integers(2, width + 1)))]
        succ[u].extend(fan)
        for v in fan:
            if rng.integers(2):
                succ[v].append(new())
        fans.append(fan)
    for a, b in zip(fans, fans[1:]):  # a join of two fans' last ops
        j = new()
        succ[a[-1]].append(j)
        succ[b[-1]].append(j)
    sink = new()
    for v in range(n - 1):
        if not succ[v]:
            succ[v].append(sink)
    ptr = np.zeros(n + 1, np.int64)
    ptr[1:] = np.cumsum([len(x) for x in succ])
    return ptr, np.array([x for l in succ for x in l], np.int32), n


def test_fans_with_delays(mlsim):
    """Fans of ops with one predecessor: chained members release each other
    at the source's output time (its finish plus its resource's delay),
    whatever their own resources and priorities; with and without gaps and a
    placement."""
    rng = np.random.default_rng(31)
    for case in range(6):
        ptr, idx, n = fan_graph(rng, int(rng.integers(1, 6)), int(rng.choice([3, 8, 13])))
        R, S = int(rng.integers(2, 7)), 131
        res = rng.integers(0, R, size=n).astype(np.int32)
        prio = rng.integers(-3, 4, size=n).astype(np.int32) if case % 2 else None
        dur = W.random_durations(n, S, 1, int(rng.choice([4, 5000])), rng)
        delay = rng.integers(0, 6000, size=R).astype(np.int32)
        gap = rng.integers(0, 2000, size=R).astype(np.int32) if case % 3 == 0 else None
        place = rng.integers(0, R, size=(n, S)).astype(np.uint16) if case % 3 == 1 else None
        print(f"fans case {case}: n={n} R={R} prio={prio is not None} gap={gap is not None} "
              f"place={place is not None}", flush=True)
        check(mlsim, ptr, idx, res, R, dur, None, None, prio=prio, place=place)
        check(mlsim, ptr, idx, res, R, dur, gap, delay, prio=prio, place=place)


def test_random_graphs_many_resources(mlsim):
    """Barriers of ops sharing predecessors, resource tables too large for
    LDS, priorities, duplicate edges, ragged tiles."""
    rng = np.random.default_rng(18)
    for n, R, p in ((60, 3, 0.1), (300, 700, 0.02), (150, 40, 0.05), (200, 5, 0.3)):
        ptr, idx, res, prio = W.random_dag(n, R, p, rng, with_prio=True, dup_edges=True)
        dur = W.random_durations(n, 97, 1, 5000, rng)
        gap = rng.integers(0, 3000, size=R).astype(np.int32)
        delay = rng.integers(0, 8000, size=R).astype(np.int32)
        print(f"random n={n} R={R}", flush=True)
        check(mlsim, ptr, idx, res, R, dur, gap, delay, prio=prio)
        check(mlsim, ptr, idx, res, R, dur, None, delay, prio=prio)


def test_barrier_members_share_the_delayed_ready_time(mlsim):
    # ops 0 (R0) and 1 (R1) both feed ops 2, 3, 4 (one shared predecessor
    # set: a barrier); R0's outputs take 7 ns, R1's 2 ns
    ptr = np.array([0, 3, 6, 6, 6, 6], np.int64)
    idx = np.array([2, 3, 4, 2, 3, 4], np.int32)
    res = np.array([0, 1, 2, 3, 2], np.int32)
    rng = np.random.default_rng(5)
    dur = rng.integers(1, 20, size=(5, 64 * 3 + 5)).astype(np.int32)
    check(mlsim, ptr, idx, res, 4, dur, None, np.array([7, 2, 0, 0], np.int32))
    check(mlsim, ptr, idx, res, 4, dur, np.array([1, 0, 3, 0], np.int32), np.array([7, 2, 50, 1], np.int32))


def test_overflow_and_bad_durations(mlsim):
    n = 4
    ptr = np.array([0, 1, 2, 3, 3], np.int64)  # a chain over two resources
    idx = np.array([1, 2, 3], np.int32)
    res = np.array([0, 1, 0, 1], np.int32)
    dur = np.full((n, 6), 2**28, np.int32)
    dur[0, 1] = 0  # bad duration
    dur[:, 2] = 1
    delay = np.array([2**29, 2**29], np.int32)  # 4 * 2^28 + 3 * 2^29 > INT32_MAX
    omk, ost = check(mlsim, ptr, idx, res, 2, dur, None, delay)
    assert ost[0] == oracle.ST_OVERFLOW and ost[1] == oracle.ST_BAD_DUR and ost[2] == 0
    # a delay past INT32_MAX after the last op alone is no overflow
    big = np.array([2**31 - 1, 2**31 - 1], np.int32)
    omk, ost = check(mlsim, np.array([0, 0, 0], np.int64), np.zeros(0, np.int32), np.array([0, 1], np.int32), 2,
                     np.full((2, 3), 2**30, np.int32), None, big)
    assert (ost == 0).all() and (omk == 2**30).all()
    # and a delay that pushes a successor's ready time to 2^31 or beyond is
    omk, ost = check(mlsim, np.array([0, 1, 1], np.int64), np.array([1], np.int32), np.array([0, 1], np.int32), 2,
                     np.full((2, 3), 2, np.int32), None, big)
    assert (ost == oracle.ST_OVERFLOW).all()


def test_bert_full_size_sampled(mlsim):
    w = W.make_config(4)
    dur = w.durations()
    gap = np.full(w.n_res, 2_000, np.int32)
    gap[: 16] = 5_000
    delay = np.full(w.n_res, 10_000, np.int32)  # link ops: the copy out of the receive buffer
    delay[: 16] = 0
    g = mlsim.Graph.from_workload(w)
    mk, fin, st = g.run(dev(dur), want_finish=True, gap=gap, delay=delay)
    torch.cuda.synchronize()
    rng = np.random.default_rng(4)
    scen = np.unique(np.r_[0, w.n_scen - 1, rng.integers(0, w.n_scen, 30)])
    sub = np.ascontiguousarray(dur[:, scen])
    omk, ofin, ost = oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, sub, gap=gap, delay=delay)
    sel = torch.from_numpy(scen).cuda()
    assert np.array_equal(mk[sel].cpu().numpy(), omk)
    assert np.array_equal(st[sel].cpu().numpy(), ost)
    assert np.array_equal(fin[:, sel].cpu().numpy(), ofin)
    g.close()


def test_arrays_read_before_return(mlsim):
    """The call has read both host arrays when it returns: overwriting them
    before the stream runs does not change the result."""
    w = W.make_config(2, n_scen=128)
    dur = w.durations()
    gap = np.full(w.n_res, 3000, np.int32)
    delay = np.full(w.n_res, 700, np.int32)
    keep_gap, keep_delay = gap.copy(), delay.copy()
    g = mlsim.Graph.from_workload(w)
    d = dev(dur)
    torch.cuda._sleep(50_000_000)  # keep the stream busy so the replay runs after the overwrite
    mk, fin, st = g.run(d, want_finish=True, gap=gap, delay=delay)
    gap[:] = 10**9
    delay[:] = 10**9
    torch.cuda.synchronize()
    omk, ofin, ost = oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur, gap=keep_gap,
                                      delay=keep_delay)
    assert np.array_equal(mk.cpu().numpy(), omk) and np.array_equal(fin.cpu().numpy(), ofin)
    g.close()
