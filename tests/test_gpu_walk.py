"""GPU parity of the lockstep walk (algo "walk") against the CPU oracle.

The walk replays every scenario of a tile along one pilot scenario's event
order and checks each scenario's schedule; scenarios that fail the check are
replayed by the event kernel.  These tests compare the final outputs with
oracle/ bit for bit, and separately count how many scenarios the walk itself
completed (the diagnostic MLSIM_WALK_NO_RETRY leaves flagged scenarios at
makespan -2), so a walk that silently flags everything cannot pass.
"""
import os

import numpy as np
import pytest

import oracle
from paper_2002_06790_amd import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

RETRY = -2


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


def run_walk(mlsim, ptr, idx, res, R, dur, prio=None, want_finish=True, ld_pad=0):
    g = mlsim.Graph(ptr, idx, res, R, prio=prio)
    eligible = g.walk_eligible()
    S = dur.shape[1]
    d = dev(np.pad(dur, ((0, 0), (0, ld_pad)))) if ld_pad else dev(dur)
    mk, fin, st = g.run(d[:, :S], want_finish=want_finish, algo="walk")
    torch.cuda.synchronize()
    g.close()
    return eligible, mk.cpu().numpy(), (fin.cpu().numpy() if want_finish else None), st.cpu().numpy()


def check(mlsim, ptr, idx, res, R, dur, prio=None, want_finish=True, ld_pad=0, need_walk=True):
    eligible, mk, fin, st = run_walk(mlsim, ptr, idx, res, R, dur, prio, want_finish, ld_pad)
    if need_walk:
        assert eligible, "graph unexpectedly outside the walk's limits"
    omk, ofin, ost = oracle.run_batch(ptr, idx, res, R, dur, prio=prio)
    assert np.array_equal(st, ost), "status differs"
    assert np.array_equal(mk, omk), f"makespan differs in {np.count_nonzero(mk != omk)} scenarios"
    if want_finish:
        ok = ost == 0
        assert np.array_equal(fin[:, ok], ofin[:, ok]), "finish times differ"


def walk_only(mlsim, monkeypatch, ptr, idx, res, R, dur, prio=None):
    """Walk without the event retry: returns the fraction of scenarios the
    walk completed, after checking that each of them equals the oracle."""
    monkeypatch.setenv("MLSIM_WALK_NO_RETRY", "1")
    try:
        eligible, mk, fin, st = run_walk(mlsim, ptr, idx, res, R, dur, prio)
    finally:
        monkeypatch.delenv("MLSIM_WALK_NO_RETRY")
    assert eligible
    omk, ofin, ost = oracle.run_batch(ptr, idx, res, R, dur, prio=prio)
    done = mk != RETRY
    assert np.array_equal(mk[done], omk[done]), "a scenario the walk accepted differs from the oracle"
    assert np.array_equal(fin[:, done], ofin[:, done]), "finish times of accepted scenarios differ"
    assert (st[done] == 0).all()
    return float(done.mean())


# ---------------------------------------------------------------- workloads

@pytest.mark.parametrize("k,S", [(1, 1024), (2, 200), (3, 333), (4, 200)])
def test_walk_workload_parity(mlsim, k, S):
    w = W.make_config(k, n_scen=S if k != 1 else None)
    dur = w.durations()
    print(f"walk workload {w.name} n={w.n_ops} S={dur.shape[1]}", flush=True)
    check(mlsim, w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur)


def test_walk_bert_all_knobs(mlsim):
    """Slices of every strategy knob of the BERT workload (different knobs
    order the resources very differently)."""
    w = W.make_config(4)
    scen = np.concatenate([np.arange(k * 4096, k * 4096 + 130) for k in range(12)])
    dur, _ = w.columns(scen)
    check(mlsim, w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur)


@pytest.mark.parametrize("k,S,floor", [(1, 1024, 0.8), (3, 2048, 0.95), (4, 2048, 0.95)])
def test_walk_completes_most_scenarios(mlsim, monkeypatch, k, S, floor):
    """The walk itself (no retry) completes most scenarios of the workloads
    whose scenarios are close to each other, and every scenario it completes
    equals the oracle."""
    w = W.make_config(k, n_scen=S if k != 1 else None)
    dur = w.durations()
    frac = walk_only(mlsim, monkeypatch, w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur)
    print(f"{w.name}: walk completed {frac:.4f} of {dur.shape[1]} scenarios", flush=True)
    assert frac >= floor


# ----------------------------------------------------------- random graphs

def test_walk_random_graphs(mlsim, monkeypatch):
    """Random DAGs with priorities, repeated edges and small duration ranges
    (many equal times); the walk's accepted scenarios equal the oracle and
    the retried ones are fixed by the event kernel."""
    rng = np.random.default_rng(31337)
    for case in range(40):
        n = int(rng.integers(1, 80))
        R = int(rng.integers(1, 9))
        S = int(rng.choice([1, 5, 63, 64, 65, 130, 200]))
        hi = int(rng.choice([2, 3, 10, 1000]))
        ptr, idx, res, pr = W.random_dag(n, R, float(rng.uniform(0, 0.3)), rng,
                                         with_prio=bool(rng.integers(2)), dup_edges=bool(rng.integers(2)))
        dur = W.random_durations(n, S, 1, hi, rng)
        print(f"walk random case {case} n={n} R={R} S={S} hi={hi}", flush=True)
        check(mlsim, ptr, idx, res, R, dur, prio=pr, ld_pad=int(rng.integers(0, 3)) * 7)
        walk_only(mlsim, monkeypatch, ptr, idx, res, R, dur, prio=pr)


def test_walk_noisy_copies(mlsim, monkeypatch):
    """Scenarios that are 1 % perturbations of one base scenario, the case the
    walk is built for: most are completed by the walk itself."""
    rng = np.random.default_rng(5)
    fracs = []
    for case in range(10):
        n, R = int(rng.integers(20, 300)), int(rng.integers(2, 12))
        ptr, idx, res, pr = W.random_dag(n, R, float(rng.uniform(0.01, 0.08)), rng, with_prio=False,
                                         dup_edges=False)
        base = rng.integers(1000, 100000, size=(n, 1)).astype(np.float64)
        dur = np.maximum(1, np.rint(base * np.exp(0.01 * rng.standard_normal((n, 256))))).astype(np.int32)
        check(mlsim, ptr, idx, res, R, dur, prio=pr)
        fracs.append(walk_only(mlsim, monkeypatch, ptr, idx, res, R, dur, prio=pr))
    print("walk completed fractions:", np.round(fracs, 3), flush=True)
    assert np.mean(fracs) > 0.5


def test_walk_barriers(mlsim, monkeypatch):
    """Groups of ops sharing a predecessor set (barrier nodes), random
    priorities and equal times."""
    from test_gpu_parity import barrier_case
    rng = np.random.default_rng(606)
    for case in range(30):
        ptr, idx, res, prio, dur = barrier_case(rng, int(rng.integers(2, 6)), int(rng.integers(1, 6)),
                                                int(rng.integers(0, 12)), int(rng.integers(1, 4)),
                                                int(rng.choice([64, 130])), int(rng.choice([1, 3, 50])))
        R = int(res.max()) + 1
        check(mlsim, ptr, idx, res, R, dur, prio=prio)
        walk_only(mlsim, monkeypatch, ptr, idx, res, R, dur, prio=prio)


def test_walk_status_and_goldens(mlsim):
    """Bad durations and overflow are flagged by the walk and reported by the
    event replay exactly as the oracle does; the worked examples match."""
    import goldens
    ptr = np.array([0, 1, 2, 2], np.int64)
    idx = np.array([1, 2], np.int32)
    res = np.zeros(3, np.int32)
    dur = np.array([[1, 0, 5, 1_500_000_000, 9, -4],
                    [1, 1, 5, 1_500_000_000, 9, 1],
                    [1, 1, 5, 1, 9, 1]], np.int32)
    check(mlsim, ptr, idx, res, 1, dur)
    for gd in goldens.all_goldens():
        check(mlsim, gd["succ_ptr"], gd["succ_idx"], gd["op_res"], gd["n_res"], gd["dur"], prio=gd["prio"])


def test_walk_makespan_only_and_repeat(mlsim):
    w = W.make_config(3, n_scen=700)
    dur = dev(w.durations())
    g = mlsim.Graph.from_workload(w)
    a = [t.clone() for t in g.run(dur, want_finish=True, algo="walk")]
    b = g.run(dur, want_finish=False, algo="walk")
    c = g.run(dur, want_finish=True, algo="event")
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0]) and torch.equal(a[2], b[2])
    assert all(torch.equal(x, y) for x, y in zip(a, c))
    g.close()
