"""GPU parity of the replay with a gap per resource (sim_run_batch_gap).

A resource that finishes an op cannot start its next op before its gap has
passed.  Every case calls the library through its C ABI and compares the
integer outputs element by element with the oracle's replay with gaps.
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


def check(mlsim, ptr, idx, res, R, dur, gap, prio=None, place=None):
    g = mlsim.Graph(ptr, idx, res, R, prio=prio)
    mk, fin, st = g.run(dev(dur), place=dev_place(place), want_finish=True, algo="event", gap=gap)
    torch.cuda.synchronize()
    omk, ofin, ost = oracle.run_batch(ptr, idx, res, R, dur, prio=prio, place=place, gap=gap)
    st = st.cpu().numpy()
    assert np.array_equal(st, ost), "status differs"
    assert np.array_equal(mk.cpu().numpy(), omk), "makespan differs"
    ok = ost == 0
    assert np.array_equal(fin.cpu().numpy()[:, ok], ofin[:, ok]), "finish times differ"
    g.close()
    return omk, ost


def test_hand_example(mlsim):
    ptr = np.array([0, 0, 1, 1, 1], np.int64)
    idx = np.array([2], np.int32)
    res = np.array([0, 1, 0, 0], np.int32)
    dur = np.array([[5], [2], [4], [1]], np.int32)
    g = mlsim.Graph(ptr, idx, res, 2)
    mk, fin, _ = g.run(dev(dur), want_finish=True, gap=[3, 0])
    torch.cuda.synchronize()
    assert fin.cpu().numpy()[:, 0].tolist() == [5, 2, 16, 9] and int(mk[0]) == 16
    g.close()


@pytest.mark.parametrize("k,S", [(1, 1024), (2, 200), (3, 333), (4, 200), (5, 130)])
def test_workload_parity(mlsim, k, S):
    w = W.make_config(k, n_scen=S if k != 1 else None)
    dur = w.durations()
    rng = np.random.default_rng(k)
    gap = rng.integers(0, 20_000, size=w.n_res).astype(np.int32)
    gap[0] = 0
    print(f"gap workload {w.name} S={dur.shape[1]}", flush=True)
    check(mlsim, w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur, gap, prio=w.prio, place=w.placement())


def test_zero_gaps_equal_plain_replay(mlsim):
    w = W.make_config(4, n_scen=256)
    dur = w.durations()
    g = mlsim.Graph.from_workload(w)
    d = dev(dur)
    mk, fin, st = g.run(d, want_finish=True, algo="event")
    gmk, gfin, gst = g.run(d, want_finish=True, gap=np.zeros(w.n_res, np.int32))
    torch.cuda.synchronize()
    assert torch.equal(mk, gmk) and torch.equal(fin, gfin) and torch.equal(st, gst)
    g.close()


def test_random_graphs_many_resources(mlsim):
    """Resource tables too large for LDS, priorities, duplicate edges, ragged tiles."""
    rng = np.random.default_rng(8)
    for n, R, p in ((60, 3, 0.1), (300, 700, 0.02), (150, 40, 0.05)):
        ptr, idx, res, prio = W.random_dag(n, R, p, rng, with_prio=True, dup_edges=True)
        dur = W.random_durations(n, 97, 1, 5000, rng)
        gap = rng.integers(0, 3000, size=R).astype(np.int32)
        print(f"random n={n} R={R}", flush=True)
        check(mlsim, ptr, idx, res, R, dur, gap, prio=prio)


def test_overflow_and_bad_durations(mlsim):
    n = 4
    ptr = np.array([0, 1, 2, 3, 3], np.int64)  # a chain on one resource
    idx = np.array([1, 2, 3], np.int32)
    res = np.zeros(n, np.int32)
    dur = np.full((n, 5), 2**28, np.int32)
    dur[0, 1] = 0  # bad duration
    dur[:, 2] = 1
    gap = np.array([2**29], np.int32)  # 4 * 2^28 + 3 * 2^29 > INT32_MAX
    omk, ost = check(mlsim, ptr, idx, res, 1, dur, gap)
    assert ost[0] == oracle.ST_OVERFLOW and ost[1] == oracle.ST_BAD_DUR and ost[2] == 0


def test_bert_full_size_sampled(mlsim):
    w = W.make_config(4)
    dur = w.durations()
    gap = np.full(w.n_res, 2_000, np.int32)
    gap[: 16] = 5_000  # compute streams: launch gaps; links: protocol gaps
    g = mlsim.Graph.from_workload(w)
    mk, fin, st = g.run(dev(dur), want_finish=True, gap=gap)
    torch.cuda.synchronize()
    rng = np.random.default_rng(4)
    scen = np.unique(np.r_[0, w.n_scen - 1, rng.integers(0, w.n_scen, 30)])
    sub = np.ascontiguousarray(dur[:, scen])
    omk, ofin, ost = oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, sub, gap=gap)
    sel = torch.from_numpy(scen).cuda()
    assert np.array_equal(mk[sel].cpu().numpy(), omk)
    assert np.array_equal(st[sel].cpu().numpy(), ost)
    assert np.array_equal(fin[:, sel].cpu().numpy(), ofin)
    g.close()


def test_gap_array_read_before_return(mlsim):
    """The call has read the host gap array when it returns: overwriting it
    before the stream runs does not change the result."""
    w = W.make_config(2, n_scen=128)
    dur = w.durations()
    gap = np.full(w.n_res, 3000, np.int32)
    keep = gap.copy()
    g = mlsim.Graph.from_workload(w)
    d = dev(dur)
    torch.cuda._sleep(50_000_000)  # keep the stream busy so the replay runs after the overwrite
    mk, fin, st = g.run(d, want_finish=True, gap=gap)
    gap[:] = 10**9
    torch.cuda.synchronize()
    omk, ofin, ost = oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur, gap=keep)
    assert np.array_equal(mk.cpu().numpy(), omk) and np.array_equal(fin.cpu().numpy(), ofin)
    g.close()
