"""GPU parity of the bottleneck attribution (sim_attribute) against the CPU oracle.

The library replays every scenario, records each op's predecessor on its
resource, sums each resource's busy time and walks each scenario's binding
chain.  busy, chain, chain_ops, makespan, status, finish and the chain of one
scenario are compared with oracle.attribute / oracle.run_batch element by
element; each op's recorded predecessor on its resource is checked against
the schedule (it is the op that ran right before on that resource).
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


def check_prev(res, dur, fin, prev, ok):
    """prev[v] is the op that ran right before v on v's resource (-1: none)."""
    n, S = dur.shape
    for s in np.flatnonzero(ok):
        r = res[:, s] if res.ndim == 2 else res
        start = fin[:, s].astype(np.int64) - dur[:, s]
        expect = np.full(n, -1, np.int64)
        for q in np.unique(r):
            ops = np.flatnonzero(r == q)
            ops = ops[np.argsort(start[ops], kind="stable")]
            expect[ops[1:]] = ops[:-1]
        assert np.array_equal(prev[:, s], expect), f"predecessor on resource differs in scenario {s}"


def check_attr(mlsim, ptr, idx, res, R, dur, prio=None, place=None, path_scen=-1, prev_cols=8):
    g = mlsim.Graph(ptr, idx, res, R, prio=prio)
    S = dur.shape[1]
    p = None
    if place is not None:
        p = torch.from_numpy(np.ascontiguousarray(place).view(np.int16)).cuda().view(torch.uint16)
    out = g.attribute(dev(dur), place=p, path_scen=path_scen)
    torch.cuda.synchronize()
    omk, ost, obusy, ochain, oops, opath = oracle.attribute(ptr, idx, res, R, dur, prio=prio, place=place,
                                                            path_scen=path_scen)
    _, ofin, _ = oracle.run_batch(ptr, idx, res, R, dur, prio=prio, place=place)
    h = {k: (v.cpu().numpy() if isinstance(v, torch.Tensor) else v) for k, v in out.items()}
    assert np.array_equal(h["status"], ost), "status differs"
    assert np.array_equal(h["makespan"], omk), "makespan differs"
    assert np.array_equal(h["busy"], obusy), "busy time differs"
    assert np.array_equal(h["chain"], ochain), "chain time differs"
    assert np.array_equal(h["chain_ops"], oops), "chain length differs"
    ok = ost == 0
    assert np.array_equal(h["finish"][:, ok], ofin[:, ok]), "finish times differ"
    if path_scen >= 0:
        assert np.array_equal(h["path"], opath), "chain of one scenario differs"
    cols = np.flatnonzero(ok)[:prev_cols]
    sel = np.zeros(S, bool)
    sel[cols] = True
    rr = place.astype(np.int64) if place is not None else np.asarray(res)
    check_prev(rr[:, sel] if place is not None else rr, dur[:, sel], h["finish"][:, sel], h["prev"][:, sel],
               np.ones(sel.sum(), bool))
    g.close()
    return h


@pytest.mark.parametrize("k,S", [(1, 1024), (2, 130), (3, 200), (4, 130), (5, 70)])
def test_attr_workloads(mlsim, k, S):
    w = W.make_config(k, n_scen=S)
    print(f"attribution workload {w.name} n={w.n_ops} S={S}", flush=True)
    check_attr(mlsim, w.succ_ptr, w.succ_idx, w.op_res, w.n_res, w.durations(), prio=w.prio,
               place=w.placement(), path_scen=S - 1)


def test_attr_placement_wide_fanout(mlsim):
    """Attribution under a placement on layered graphs whose ops have up to
    24 successors (the placement replay's grouped successor entries, with
    predecessor recording)."""
    from test_gpu_parity import wide_layered
    rng = np.random.default_rng(1618)
    for case, (levels, width, max_in) in enumerate([(6, 24, 12), (5, 20, 20)]):
        ptr, idx = wide_layered(rng, levels, width, max_in)
        n, R, S = levels * width, int(rng.integers(2, 9)), 70
        print(f"case {case}: n={n} R={R} S={S} max out-degree {np.diff(ptr).max()}", flush=True)
        res = rng.integers(0, R, size=n).astype(np.int32)
        dur = W.random_durations(n, S, 1, int(rng.choice([3, 5000])), rng)
        place = rng.integers(0, R, size=(n, S)).astype(np.uint16)
        check_attr(mlsim, ptr, idx, res, R, dur, place=place, path_scen=S - 1)


def test_attr_random_graphs(mlsim):
    """Random DAGs with priorities, repeated edges, placement and small
    duration ranges (many equal times, so the tie rules matter)."""
    rng = np.random.default_rng(2718)
    for case in range(40):
        n = int(rng.integers(1, 80))
        R = int(rng.integers(1, 9))
        S = int(rng.choice([1, 5, 63, 64, 65, 130]))
        ptr, idx, res, pr = W.random_dag(n, R, float(rng.uniform(0, 0.3)), rng,
                                         with_prio=bool(rng.integers(2)), dup_edges=bool(rng.integers(2)))
        dur = W.random_durations(n, S, 1, int(rng.choice([2, 3, 10, 1000])), rng)
        place = rng.integers(0, R, size=(n, S)).astype(np.uint16) if rng.integers(3) == 0 else None
        print(f"attribution random case {case} n={n} R={R} S={S}", flush=True)
        check_attr(mlsim, ptr, idx, res, R, dur, prio=pr, place=place, path_scen=int(rng.integers(S)))


@pytest.mark.parametrize("groups", [1, 2])
def test_attr_heap_children_in_registers(mlsim, groups, pin_variants):
    """The recording replay with the heap root's children in registers
    (chosen by the launcher when the chip is full; forced here)."""
    pin_variants(ev_reg=1, ev_lds_groups=groups)
    for k, S in ((4, 130), (2, 70), (1, 1024)):
        w = W.make_config(k, n_scen=S)
        check_attr(mlsim, w.succ_ptr, w.succ_idx, w.op_res, w.n_res, w.durations(), prio=w.prio,
                   path_scen=S - 1)
    rng = np.random.default_rng(2719)
    for case in range(10):
        n, R, S = int(rng.integers(1, 80)), int(rng.integers(1, 9)), int(rng.choice([1, 65, 130]))
        ptr, idx, res, pr = W.random_dag(n, R, float(rng.uniform(0, 0.3)), rng, with_prio=True)
        dur = W.random_durations(n, S, 1, int(rng.choice([3, 1000])), rng)
        check_attr(mlsim, ptr, idx, res, R, dur, prio=pr, path_scen=int(rng.integers(S)))


def test_attr_wide_rows(mlsim):
    """A graph with more ops than 16-bit rows can name (70000): the last-op
    table keeps 32-bit rows; checked against the oracle on a few scenarios."""
    rng = np.random.default_rng(65536)
    n, R = 70000, 8
    # op v > 0 takes one or two predecessors among the 64 ops before it
    v = np.repeat(np.arange(1, n), 2)
    u = v - rng.integers(1, 65, size=v.size)
    keep = (u >= 0) & ((np.arange(v.size) % 2 == 0) | (rng.random(v.size) < 0.5))
    u, v = u[keep], v[keep]
    order = np.lexsort((v, u))
    u, v = u[order], v[order]
    ptr = np.zeros(n + 1, np.int64)
    np.add.at(ptr, u + 1, 1)
    ptr = np.cumsum(ptr)
    idx = v.astype(np.int32)
    res = rng.integers(0, R, size=n).astype(np.int32)
    dur = W.random_durations(n, 70, 1, 1000, rng)
    print(f"attribution on {n} ops", flush=True)
    check_attr(mlsim, ptr, idx, res, R, dur, path_scen=3)


def test_attr_status_and_empty(mlsim):
    ptr = np.array([0, 1, 2, 2], np.int64)
    idx = np.array([1, 2], np.int32)
    res = np.zeros(3, np.int32)
    dur = np.array([[1, 0, 5, 1_500_000_000, 9, -4],
                    [1, 1, 5, 1_500_000_000, 9, 1],
                    [1, 1, 5, 1, 9, 1]], np.int32)
    h = check_attr(mlsim, ptr, idx, res, 1, dur, path_scen=1)
    assert h["path"].tolist() == []
    g0 = mlsim.Graph(np.zeros(1, np.int64), np.zeros(0, np.int32), np.zeros(0, np.int32), 2)
    out = g0.attribute(torch.zeros((0, 9), dtype=torch.int32, device="cuda"), path_scen=3)
    torch.cuda.synchronize()
    for k in ("makespan", "status", "chain_ops", "busy", "chain"):
        assert (out[k].cpu().numpy() == 0).all(), k
    assert out["path"].tolist() == []
    g0.close()


def test_attr_full_size_sampled(mlsim):
    """The BERT workload at its full scenario count; sampled scenarios
    against the oracle, every scenario's chain summing to its makespan."""
    w = W.make_config(4)
    dur_h = w.durations()
    g = mlsim.Graph.from_workload(w)
    out = g.attribute(dev(dur_h), path_scen=w.n_scen - 1)
    torch.cuda.synchronize()
    mk = out["makespan"].cpu().numpy()
    assert (out["status"].cpu().numpy() == 0).all()
    assert np.array_equal(out["chain"].sum(0, dtype=torch.int64).cpu().numpy(), mk.astype(np.int64))
    rng = np.random.default_rng(505)
    scen = np.unique(np.r_[0, w.n_scen - 1, rng.integers(0, w.n_scen, 40)])
    omk, ost, obusy, ochain, oops, opath = oracle.attribute(w.succ_ptr, w.succ_idx, w.op_res, w.n_res,
                                                            dur_h[:, scen], path_scen=scen.size - 1)
    sel = torch.from_numpy(scen).cuda()
    assert np.array_equal(mk[scen], omk)
    assert np.array_equal(out["busy"][:, sel].cpu().numpy(), obusy)
    assert np.array_equal(out["chain"][:, sel].cpu().numpy(), ochain)
    assert np.array_equal(out["chain_ops"][sel].cpu().numpy(), oops)
    assert np.array_equal(out["path"], opath)
    g.close()
