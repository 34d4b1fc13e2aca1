"""GPU parity of the static-order replay (sim_static_*) against the CPU oracle.

Every device runs its ops in a given order; the library compiles the order
into a max-plus sweep and runs it on the GPU.  Outputs are compared with
oracle.static_run element by element; with the event replay's own run order
the result must also equal the event replay of that scenario.
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


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dtype=torch.int32, device="cuda")


def event_order(dur_col, fin_col):
    """All ops by start time in a replay (ties by op id): each device's part
    is the order in which that device ran its ops."""
    start = fin_col.astype(np.int64) - dur_col
    return np.lexsort((np.arange(dur_col.size), start)).astype(np.int32)


def random_linear_extension(n, ptr, idx, rng):
    """A random topological order of the DAG (any such order is a valid run
    order for every device)."""
    cnt = np.zeros(n, np.int64)
    np.add.at(cnt, idx, 1)
    ready = [v for v in range(n) if cnt[v] == 0]
    out = []
    while ready:
        v = ready.pop(int(rng.integers(len(ready))))
        out.append(v)
        for e in range(ptr[v], ptr[v + 1]):
            w = int(idx[e])
            cnt[w] -= 1
            if cnt[w] == 0:
                ready.append(w)
    assert len(out) == n
    return np.array(out, np.int32)


def check_static(mlsim, ptr, idx, res, R, order, dur, want_finish=True, ld_pad=0, prio=None):
    g = mlsim.Graph(ptr, idx, res, R, prio=prio)
    st_obj = g.static_order(order)
    S = dur.shape[1]
    d = dev(np.pad(dur, ((0, 0), (0, ld_pad)))) if ld_pad else dev(dur)
    mk, fin, st = st_obj.run(d[:, :S], want_finish=want_finish)
    torch.cuda.synchronize()
    omk, ofin, ost = oracle.static_run(ptr, idx, res, R, order, dur)
    assert np.array_equal(st.cpu().numpy(), ost), "status differs"
    assert np.array_equal(mk.cpu().numpy(), omk), "makespan differs"
    if want_finish:
        ok = ost == 0
        assert np.array_equal(fin.cpu().numpy()[:, ok], ofin[:, ok]), "finish times differ"
    st_obj.close()
    g.close()
    return omk, ofin


@pytest.mark.parametrize("k,S", [(1, 1024), (2, 130), (3, 200), (4, 130), (5, 70)])
def test_static_workloads_event_order(mlsim, k, S):
    """Each workload with the run order the event replay chose in its first
    scenario: every scenario against the oracle, and the first scenario
    against the event replay itself."""
    w = W.make_config(k, n_scen=S)
    dur = w.durations()
    place = w.placement()
    res = w.op_res if place is None else place[:, 0].astype(np.int32)
    print(f"static workload {w.name} n={w.n_ops} S={S}", flush=True)
    emk, efin, _ = oracle.run_batch(w.succ_ptr, w.succ_idx, res, w.n_res, dur[:, :1], prio=w.prio)
    order = event_order(dur[:, 0], efin[:, 0])
    omk, ofin = check_static(mlsim, w.succ_ptr, w.succ_idx, res, w.n_res, order, dur, prio=w.prio)
    assert omk[0] == emk[0] and np.array_equal(ofin[:, 0], efin[:, 0])


def test_static_random_orders(mlsim):
    """Random DAGs with random linear extensions as run orders, scenario
    counts around the wavefront width, padded leading dimensions, finish
    times on and off."""
    rng = np.random.default_rng(8080)
    for case in range(40):
        n = int(rng.integers(1, 90))
        R = int(rng.integers(1, 9))
        S = int(rng.choice([1, 5, 63, 64, 65, 130]))
        ptr, idx, res, _ = W.random_dag(n, R, float(rng.uniform(0, 0.3)), rng, with_prio=False,
                                        dup_edges=bool(rng.integers(2)))
        dur = W.random_durations(n, S, 1, int(rng.choice([3, 1000])), rng)
        order = random_linear_extension(n, ptr, idx, rng)
        print(f"static random case {case} n={n} R={R} S={S}", flush=True)
        check_static(mlsim, ptr, idx, res, R, order, dur, want_finish=bool(rng.integers(2)),
                     ld_pad=int(rng.integers(0, 3)) * 5)


@pytest.mark.parametrize("slots", ["lds", "global"])
def test_static_wide_graphs(mlsim, slots, pin_variants):
    """Wide layers keep many values live; value slots in LDS where they fit
    or in global scratch."""
    if slots == "global":
        pin_variants(cp_global=1)
    rng = np.random.default_rng(99)
    for case in range(3):
        n = 900
        ptr, idx, res, _ = W.random_dag(n, 4, 0.004, rng, with_prio=False, dup_edges=False)
        dur = W.random_durations(n, 100, 1, 1000, rng)
        order = random_linear_extension(n, ptr, idx, rng)
        check_static(mlsim, ptr, idx, res, 4, order, dur)


def test_static_status_errors_and_empty(mlsim):
    ptr = np.array([0, 1, 2, 2], np.int64)
    idx = np.array([1, 2], np.int32)
    res = np.zeros(3, np.int32)
    dur = np.array([[1, 0, 5, 1_500_000_000, 9, -4],
                    [1, 1, 5, 1_500_000_000, 9, 1],
                    [1, 1, 5, 1, 9, 1]], np.int32)
    check_static(mlsim, ptr, idx, res, 1, np.array([0, 1, 2], np.int32), dur)
    g = mlsim.Graph(ptr, idx, res, 1)
    for bad in ([0, 0, 1], [0, 1, 3]):
        with pytest.raises(mlsim.SimError) as e:
            g.static_order(np.array(bad, np.int32))
        assert e.value.code == mlsim.SIM_E_INVAL
    with pytest.raises(mlsim.SimError) as e:
        g.static_order(np.array([1, 0, 2], np.int32))
    assert e.value.code == mlsim.SIM_E_CYCLE
    g.close()
    g0 = mlsim.Graph(np.zeros(1, np.int64), np.zeros(0, np.int32), np.zeros(0, np.int32), 1)
    s0 = g0.static_order(np.zeros(0, np.int32))
    mk, _, st = s0.run(torch.zeros((0, 7), dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()
    assert (mk.cpu().numpy() == 0).all() and (st.cpu().numpy() == 0).all()
    s0.close()
    g0.close()


def test_static_full_size_sampled(mlsim):
    """The BERT workload at its full scenario count, finish times on;
    sampled scenarios against the oracle."""
    w = W.make_config(4)
    dur_h = w.durations()
    emk, efin, _ = oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur_h[:, :1])
    order = event_order(dur_h[:, 0], efin[:, 0])
    g = mlsim.Graph.from_workload(w)
    st_obj = g.static_order(order)
    mk, fin, st = st_obj.run(dev(dur_h), want_finish=True)
    torch.cuda.synchronize()
    rng = np.random.default_rng(404)
    scen = np.unique(np.r_[0, w.n_scen - 1, rng.integers(0, w.n_scen, 40)])
    omk, ofin, ost = oracle.static_run(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, order, dur_h[:, scen])
    sel = torch.from_numpy(scen).cuda()
    assert np.array_equal(mk[sel].cpu().numpy(), omk)
    assert np.array_equal(st[sel].cpu().numpy(), ost)
    assert np.array_equal(fin[:, sel].cpu().numpy(), ofin)
    assert mk[0].item() == emk[0]
    st_obj.close()
    g.close()
