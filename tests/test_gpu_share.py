"""GPU parity of the replay with bandwidth sharing (sim_run_batch_share).

On a shared resource every ready op starts at once and the active ops divide
its rate equally, in integer ns (see include/mlsim.h).  Every case calls the
library through its C ABI and compares the integer outputs element by
element with the oracle's sharing replay.
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


def check(mlsim, ptr, idx, res, R, dur, share, prio=None):
    g = mlsim.Graph(ptr, idx, res, R, prio=prio)
    mk, fin, st = g.run_share(dev(dur), share, want_finish=True)
    torch.cuda.synchronize()
    omk, ofin, ost = oracle.run_batch_share(ptr, idx, res, R, dur, share=share, prio=prio)
    st = st.cpu().numpy()
    assert np.array_equal(st, ost), "status differs"
    assert np.array_equal(mk.cpu().numpy(), omk), "makespan differs"
    ok = ost == 0
    assert np.array_equal(fin.cpu().numpy()[:, ok], ofin[:, ok]), "finish times differ"
    g.close()
    return omk, ost


def test_hand_examples(mlsim):
    g = mlsim.Graph(np.array([0, 0, 1, 1], np.int64), np.array([2], np.int32), np.array([0, 1, 0], np.int32), 2)
    mk, fin, _ = g.run_share(dev(np.array([[10], [4], [2]])), [1, 0], want_finish=True)
    torch.cuda.synchronize()
    assert fin.cpu().numpy()[:, 0].tolist() == [12, 4, 8] and int(mk[0]) == 12
    g.close()
    # finishes on a shared resource come before ready ops at the same time
    g = mlsim.Graph(np.array([0, 1, 1, 2, 2, 2], np.int64), np.array([3, 4], np.int32),
                    np.array([0, 0, 1, 2, 2], np.int32), 3)
    mk, fin, _ = g.run_share(dev(np.array([[2], [2], [4], [5], [5]])), [1, 0, 0], want_finish=True)
    torch.cuda.synchronize()
    assert fin.cpu().numpy()[:, 0].tolist() == [4, 4, 4, 9, 14]
    g.close()


def test_simultaneous_start_many_ops(mlsim):
    """Up to the limit of active ops, ragged tiles, counts that do not divide the unit."""
    rng = np.random.default_rng(61)
    for k in (2, 16, 17, 25, 64, 65):
        dur = rng.integers(1, 100_000, size=(k, 130)).astype(np.int32)
        check(mlsim, np.zeros(k + 1, np.int64), np.zeros(0, np.int32), np.zeros(k, np.int32), 1, dur,
              np.array([1], np.uint8))


def test_random_graphs(mlsim):
    """Shared and exclusive resources, priorities, duplicate edges, barriers."""
    rng = np.random.default_rng(62)
    for n, R, p in ((12, 2, 0.3), (60, 3, 0.1), (200, 6, 0.05), (150, 40, 0.05), (300, 4, 0.3)):
        ptr, idx, res, prio = W.random_dag(n, R, p, rng, with_prio=True, dup_edges=True)
        dur = W.random_durations(n, 97, 1, 5000, rng)
        share = (rng.random(R) < 0.5).astype(np.uint8)
        share[0] = 1
        print(f"random n={n} R={R} shared={int(share.sum())}", flush=True)
        check(mlsim, ptr, idx, res, R, dur, share, prio=prio)


@pytest.mark.parametrize("k,S", [(1, 1024), (2, 200), (3, 333), (4, 200)])
def test_workload_parity(mlsim, k, S):
    w = W.make_config(k, n_scen=S if k != 1 else None)
    dur = w.durations()
    share = np.zeros(w.n_res, np.uint8)
    share[W.link_resources(w)] = 1
    print(f"share workload {w.name} S={dur.shape[1]}", flush=True)
    omk, ost = check(mlsim, w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur, share, prio=w.prio)
    assert (ost == 0).all()


def test_key_words_without_the_resource(mlsim, pin_variants):
    """Ready-op key words holding only the op id (the layout for graphs whose
    ids and resources do not fit 32 bits together; pinned here): the
    resource then comes from the op's record, with the same results."""
    pin_variants(share_key_id=1)
    for k, S in ((4, 130), (2, 70)):
        w = W.make_config(k, n_scen=S)
        share = np.zeros(w.n_res, np.uint8)
        share[W.link_resources(w)] = 1
        print(f"share workload {w.name} S={S}, id-only key words", flush=True)
        check(mlsim, w.succ_ptr, w.succ_idx, w.op_res, w.n_res, w.durations(), share, prio=w.prio)
    rng = np.random.default_rng(63)
    for n, R, p in ((60, 3, 0.1), (200, 6, 0.05)):
        ptr, idx, res, prio = W.random_dag(n, R, p, rng, with_prio=True, dup_edges=True)
        share = (rng.random(R) < 0.5).astype(np.uint8)
        share[0] = 1
        check(mlsim, ptr, idx, res, R, W.random_durations(n, 97, 1, 5000, rng), share, prio=prio)


def test_nothing_shared_is_the_plain_replay(mlsim):
    w = W.make_config(4, n_scen=256)
    dur = dev(w.durations())
    g = mlsim.Graph.from_workload(w)
    mk, fin, st = g.run(dur, want_finish=True, algo="event")
    smk, sfin, sst = g.run_share(dur, np.zeros(w.n_res, np.uint8), want_finish=True)
    torch.cuda.synchronize()
    assert torch.equal(mk, smk) and torch.equal(fin, sfin) and torch.equal(st, sst)
    g.close()


def test_overflow_limit_and_bad_durations(mlsim):
    k = 3
    dur = np.full((k, 4), 2**30 + 1, np.int32)  # three shared ops: all end past INT32_MAX
    dur[:, 1] = 7
    dur[1, 2] = 0
    omk, ost = check(mlsim, np.zeros(k + 1, np.int64), np.zeros(0, np.int32), np.zeros(k, np.int32), 1, dur,
                     np.array([1], np.uint8))
    assert ost.tolist() == [oracle.ST_OVERFLOW, 0, oracle.ST_BAD_DUR, oracle.ST_OVERFLOW]


def test_bert_sampled_scenarios(mlsim):
    """BERT with both link directions shared (up to 25 pushes at once on an
    uplink) on 2048 scenarios; the oracle checks a sample."""
    w = W.make_config(4, n_scen=2048)
    dur = w.durations()
    share = np.zeros(w.n_res, np.uint8)
    share[W.link_resources(w)] = 1
    g = mlsim.Graph.from_workload(w)
    mk, fin, st = g.run_share(dev(dur), share, want_finish=True)
    torch.cuda.synchronize()
    rng = np.random.default_rng(6)
    scen = np.unique(np.r_[0, w.n_scen - 1, rng.integers(0, w.n_scen, 14)])
    sub = np.ascontiguousarray(dur[:, scen])
    omk, ofin, ost = oracle.run_batch_share(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, sub, share=share, prio=w.prio)
    sel = torch.from_numpy(scen).cuda()
    assert (ost == 0).all()
    assert np.array_equal(mk[sel].cpu().numpy(), omk)
    assert np.array_equal(st[sel].cpu().numpy(), ost)
    assert np.array_equal(fin[:, sel].cpu().numpy(), ofin)
    assert (st.cpu().numpy() == 0).all()
    g.close()


def test_deep_event_heap(mlsim):
    """A thousand ops ready at once: the event heap reaches far below its
    levels kept in LDS."""
    rng = np.random.default_rng(63)
    n, R = 1000, 40
    res = (np.arange(n) % R).astype(np.int32)
    ptr = np.zeros(n + 1, np.int64)
    dur = rng.integers(1, 10_000, size=(n, 70)).astype(np.int32)
    share = np.zeros(R, np.uint8)
    share[::2] = 1
    omk, ost = check(mlsim, ptr, np.zeros(0, np.int32), res, R, dur, share)
    assert (ost == 0).all()
    # and with dependencies: 10 layers of 100, each op after two of the layer before
    succ = [[] for _ in range(n)]
    for v in range(100, n):
        for u in rng.choice(np.arange(v - v % 100 - 100, v - v % 100), 2, replace=False):
            succ[u].append(v)
    ptr = np.r_[0, np.cumsum([len(x) for x in succ])].astype(np.int64)
    idx = np.array([v for x in succ for v in x], np.int32)
    check(mlsim, ptr, idx, res, R, dur, share, prio=rng.integers(-3, 4, size=n).astype(np.int32))


def test_bert_bench_launch_sampled(mlsim):
    """The benchmark's launch: BERT with its 32 links shared on all 262144
    scenarios (a persistent grid taking several rounds of tiles); sampled
    scenarios from the first and last rounds against the oracle."""
    w = W.make_config(4)
    dur = w.durations()
    share = np.zeros(w.n_res, np.uint8)
    share[W.link_resources(w)] = 1
    g = mlsim.Graph.from_workload(w)
    d = dev(dur)
    mk, fin, st = g.run_share(d, share, want_finish=True)
    torch.cuda.synchronize()
    rng = np.random.default_rng(7)
    scen = np.unique(np.r_[0, 63, 64, w.n_scen - 1, rng.integers(0, w.n_scen, 12)])
    sub = np.ascontiguousarray(dur[:, scen])
    omk, ofin, ost = oracle.run_batch_share(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, sub, share=share, prio=w.prio)
    sel = torch.from_numpy(scen).cuda()
    assert (ost == 0).all() and (st.cpu().numpy() == 0).all()
    assert np.array_equal(mk[sel].cpu().numpy(), omk)
    assert np.array_equal(fin[:, sel].cpu().numpy(), ofin)
    # a second call on the same graph (scratch already allocated) gives the same result
    mk2, _, _ = g.run_share(d, share)
    torch.cuda.synchronize()
    assert torch.equal(mk, mk2)
    g.close()


def test_first_call_captured_in_a_graph(mlsim):
    """The graph's first sharing call is captured in a HIP graph (its scratch
    exists from creation, so the call allocates nothing); every replay, with
    new durations written between replays, equals the eager call and the
    oracle."""
    w = W.make_config(4, n_scen=130)
    share = np.zeros(w.n_res, np.uint8)
    share[W.link_resources(w)] = 1
    G = mlsim.Graph.from_workload(w)
    rng = np.random.default_rng(17)
    durs = [w.durations()] + [np.maximum(1, w.durations() + rng.integers(-3000, 3000, size=(w.n_ops, 130)))
                              .astype(np.int32) for _ in range(2)]
    d = dev(durs[0])
    mk = torch.empty(130, dtype=torch.int32, device="cuda")
    st = torch.empty(130, dtype=torch.int32, device="cuda")
    fin = torch.empty((w.n_ops, 130), dtype=torch.int32, device="cuda")
    # the kernels' code is loaded by a call on another graph, outside the capture
    other = mlsim.Graph.from_workload(W.make_config(1, n_scen=64))
    other.run_share(dev(W.make_config(1, n_scen=64).durations()), [0, 0, 1])
    torch.cuda.synchronize()
    other.close()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        G.run_share(d, share, makespan=mk, finish=fin, status=st)
    for rep in range(3):
        dh = durs[rep]
        d.copy_(torch.from_numpy(dh))
        graph.replay()
        torch.cuda.synchronize()
        emk, efin, est = G.run_share(d, share, want_finish=True)
        torch.cuda.synchronize()
        assert torch.equal(mk, emk) and torch.equal(fin, efin) and torch.equal(st, est), rep
        omk, ofin, ost = oracle.run_batch_share(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dh, share=share)
        assert np.array_equal(mk.cpu().numpy(), omk) and np.array_equal(st.cpu().numpy(), ost), rep
        assert np.array_equal(fin.cpu().numpy(), ofin), rep
    G.close()
