"""GPU parity: the HIP replay equals the CPU oracle bit for bit.

Every case calls the library through its C ABI (via the ctypes binding) on
seeded inputs and compares integer nanosecond outputs element by element with
oracle/ on the same inputs.
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


def check_run(mlsim, ptr, idx, res, R, dur, prio=None, place=None, algo="event", ld_pad=0,
              want_finish=True):
    g = mlsim.Graph(ptr, idx, res, R, prio=prio)
    n, S = dur.shape
    d = dev(np.pad(dur, ((0, 0), (0, ld_pad)))) if ld_pad else dev(dur)
    d = d[:, :S]
    p = None
    if place is not None:
        p = torch.from_numpy(np.ascontiguousarray(place).view(np.int16)).cuda().view(torch.uint16)
    mk, fin, st = g.run(d, place=p, want_finish=want_finish, algo=algo)
    torch.cuda.synchronize()
    omk, ofin, ost = oracle.run_batch(ptr, idx, res, R, dur, prio=prio, place=place)
    mk, st = mk.cpu().numpy(), st.cpu().numpy()
    assert np.array_equal(st, ost), "status differs"
    assert np.array_equal(mk, omk), f"makespan differs in {np.count_nonzero(mk != omk)} scenarios"
    if want_finish:
        fin = fin.cpu().numpy()
        ok = ost == 0
        assert np.array_equal(fin[:, ok], ofin[:, ok]), "finish times differ"
    g.close()
    return omk


def check_cp(mlsim, ptr, idx, res, R, dur, paths=()):
    g = mlsim.Graph(ptr, idx, res, R)
    n, S = dur.shape
    d = dev(dur)
    cp, _ = g.critical_path(d)
    torch.cuda.synchronize()
    ocp, _ = oracle.critical_path(ptr, idx, n, dur)
    assert np.array_equal(cp.cpu().numpy(), ocp)
    for s in paths:
        _, path = g.critical_path(d, path_scen=s)
        _, opath = oracle.critical_path(ptr, idx, n, dur, path_scen=s)
        assert np.array_equal(path, opath), f"path of scenario {s}"
    g.close()


# ---------------------------------------------------------------- workloads

@pytest.mark.parametrize("k,S", [(1, 1024), (2, 200), (3, 333), (4, 200), (5, 130)])
def test_workload_parity(mlsim, k, S):
    w = W.make_config(k, n_scen=S if k != 1 else None)
    dur = w.durations()
    place = w.placement()
    print(f"workload {w.name} n={w.n_ops} S={dur.shape[1]}", flush=True)
    check_run(mlsim, w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur, place=place)
    check_cp(mlsim, w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur, paths=(0, dur.shape[1] - 1))


def test_compact_records_resource_by_row(mlsim):
    """Graphs whose key word holds the op id and first join but has no room
    for the resource (random-layered: 20000 ops, 14894 joins, 100 resources;
    a random DAG on 1000 resources): without a placement the replay reads
    each op's resource by row, with one it uses the placement."""
    w = W.make_config(5, n_scen=130)
    dur = w.durations()
    print("random-layered without placement", flush=True)
    check_run(mlsim, w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur)
    rng = np.random.default_rng(31337)
    n, R = 3000, 1000
    ptr, idx, res, _ = W.random_dag(n, R, 0.002, rng, with_prio=False)
    dur = W.random_durations(n, 100, 1, 1000, rng)
    print("random DAG on 1000 resources", flush=True)
    check_run(mlsim, ptr, idx, res, R, dur)
    place = rng.integers(0, R, size=(n, 100)).astype(np.uint16)
    check_run(mlsim, ptr, idx, res, R, dur, place=place)


def test_bert_all_knobs(mlsim):
    """Sampled scenarios of every strategy knob of the BERT workload."""
    w = W.make_config(4)
    scen = np.concatenate([np.arange(k * 4096, k * 4096 + 40) for k in range(12)])
    dur, _ = w.columns(scen)
    check_run(mlsim, w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur)


# ----------------------------------------------------------- random graphs

def rand_case(rng, n, R, p, prio, dup, S, lo=1, hi=1000):
    ptr, idx, res, pr = W.random_dag(n, R, p, rng, with_prio=prio, dup_edges=dup)
    dur = W.random_durations(n, S, lo, hi, rng)
    return ptr, idx, res, pr, dur


def test_random_graphs(mlsim):
    rng = np.random.default_rng(2024)
    for case in range(40):
        n = int(rng.integers(1, 70))
        R = int(rng.integers(1, 9))
        S = int(rng.choice([1, 5, 63, 64, 65, 130]))
        hi = int(rng.choice([3, 10, 1000]))  # small ranges force ties
        ptr, idx, res, pr, dur = rand_case(rng, n, R, float(rng.uniform(0, 0.3)),
                                           bool(rng.integers(2)), bool(rng.integers(2)), S, 1, hi)
        print(f"random case {case} n={n} R={R} S={S}", flush=True)
        check_run(mlsim, ptr, idx, res, R, dur, prio=pr, ld_pad=int(rng.integers(0, 3)) * 7)
        check_cp(mlsim, ptr, idx, res, R, dur, paths=(0,))


def wide_layered(rng, levels, width, max_in):
    """Levels of `width` ops, each op past the first fed by 1..max_in distinct
    ops of the previous level: out-degrees up to `width`, every edge direct
    (a layered graph has no longer path between consecutive levels), mixing
    joins with ops of one predecessor.  Returns (succ_ptr, succ_idx)."""
    succ = [[] for _ in range(levels * width)]
    for L in range(1, levels):
        for v in range(L * width, (L + 1) * width):
            k = int(rng.integers(1, max_in + 1))
            for u in rng.choice(width, size=k, replace=False):
                succ[(L - 1) * width + int(u)].append(v)
    ptr = np.zeros(len(succ) + 1, np.int64)
    ptr[1:] = np.cumsum([len(x) for x in succ])
    idx = np.array([x for l in succ for x in l], np.int32)
    return ptr, idx


def test_placement_wide_fanout(mlsim):
    """Ops with up to 24 successors under a placement: the placement replay
    takes an op's first eight entries as one group and the rest one at a
    time, so lanes whose ops have 0, 1, 2, 8, 9 and many more successors
    (joins and ops with a single predecessor among them) meet in one
    wavefront.  Ragged scenario count; priorities on every other case."""
    rng = np.random.default_rng(2411)
    for case, (levels, width, max_in) in enumerate([(6, 24, 12), (12, 16, 8), (4, 24, 24), (9, 12, 9)]):
        ptr, idx = wide_layered(rng, levels, width, max_in)
        n, R, S = levels * width, int(rng.integers(2, 9)), 131
        deg = np.diff(ptr)
        print(f"case {case}: n={n} R={R} S={S} max out-degree {deg.max()}", flush=True)
        assert deg.max() > 8
        res = rng.integers(0, R, size=n).astype(np.int32)
        pr = rng.integers(-3, 4, size=n).astype(np.int32) if case % 2 else None
        dur = W.random_durations(n, S, 1, 5000, rng)
        place = rng.integers(0, R, size=(n, S)).astype(np.uint16)
        check_run(mlsim, ptr, idx, res, R, dur, prio=pr, place=place)


def test_barrier_member_with_fan(mlsim):
    """Ops sharing a predecessor set (barrier members: each but the last
    releases the next through a sibling entry, first in its list) whose own
    successors form a fan of ops with a single predecessor (chained too).
    Ids are laid out so that the fan's ids fall below and above the next
    member's, with and without priorities, gaps and delays."""
    rng = np.random.default_rng(77)
    for case in range(8):
        k = int(rng.integers(3, 7))  # fan size of the first member
        # ids: fan ops, then the sources and the members (or the reverse)
        low_fans = case % 2 == 0
        nf, nm = k + 2, 3
        fan_ids = list(range(nf)) if low_fans else list(range(2 + nm, 2 + nm + nf))
        base = nf if low_fans else 0
        a, b = base, base + 1
        mem = [base + 2 + i for i in range(nm)]
        n = nf + 2 + nm
        succ = [[] for _ in range(n)]
        for m in mem:
            succ[a].append(m)
            succ[b].append(m)
        succ[mem[0]] = fan_ids[:k]                  # the fan
        succ[mem[1]] = fan_ids[k:]                  # two more ops with one predecessor
        for f in fan_ids[:k:2]:                     # some fan ops also feed one of those (a join)
            succ[f].append(fan_ids[-1])
        ptr = np.zeros(n + 1, np.int64)
        ptr[1:] = np.cumsum([len(x) for x in succ])
        idx = np.array([x for l in succ for x in l], np.int32)
        R = int(rng.integers(1, 4))
        res = rng.integers(0, R, size=n).astype(np.int32)
        pr = rng.integers(-2, 3, size=n).astype(np.int32) if case % 4 >= 2 else None
        dur = W.random_durations(n, 67, 1, int(rng.choice([3, 900])), rng)
        print(f"case {case}: n={n} fan {k} low ids {low_fans} prio {pr is not None}", flush=True)
        check_run(mlsim, ptr, idx, res, R, dur, prio=pr)
        g = mlsim.Graph(ptr, idx, res, R, prio=pr)
        gap = rng.integers(0, 50, size=R).astype(np.int32)
        delay = rng.integers(0, 50, size=R).astype(np.int32)
        mk, fin, st = g.run(dev(dur), want_finish=True, gap=gap, delay=delay)
        torch.cuda.synchronize()
        omk, ofin, ost = oracle.run_batch(ptr, idx, res, R, dur, prio=pr, gap=gap, delay=delay)
        assert np.array_equal(st.cpu().numpy(), ost) and np.array_equal(mk.cpu().numpy(), omk)
        assert np.array_equal(fin.cpu().numpy(), ofin)
        g.close()


def test_random_with_placement(mlsim):
    rng = np.random.default_rng(7)
    for _ in range(10):
        n, R, S = int(rng.integers(2, 60)), int(rng.integers(1, 12)), 97
        ptr, idx, res, pr, dur = rand_case(rng, n, R, 0.1, True, False, S, 1, 50)
        place = rng.integers(0, R, size=(n, S)).astype(np.uint16)
        check_run(mlsim, ptr, idx, res, R, dur, prio=pr, place=place)


def test_wide_and_deep_shapes(mlsim):
    rng = np.random.default_rng(8)
    # no edges, many sources (heap at its bound), one resource and many resources
    for n, R in ((300, 1), (300, 7), (257, 257)):
        ptr = np.zeros(n + 1, np.int64)
        check_run(mlsim, ptr, np.zeros(0, np.int32), rng.integers(0, R, n).astype(np.int32), R,
                  W.random_durations(n, 70, 1, 20, rng))
    # a long chain
    n = 2000
    ptr = np.arange(n + 1, dtype=np.int64).clip(max=n - 1)
    idx = np.arange(1, n, dtype=np.int32)
    ptr = np.concatenate([[0], np.cumsum(np.r_[np.ones(n - 1), 0])]).astype(np.int64)
    check_run(mlsim, ptr, idx, rng.integers(0, 3, n).astype(np.int32), 3,
              W.random_durations(n, 65, 1, 1000, rng))
    check_cp(mlsim, ptr, idx, np.zeros(n, np.int32), 1, W.random_durations(n, 65, 1, 1000, rng), (3,))


def barrier_case(rng, n_src, groups, n_free, R, S, hi):
    """Sources, then groups of ops that share one predecessor set of two or
    more sources (each group waits on one barrier), then free ops with a
    single predecessor; random priorities interleave the groups' members with
    each other and with free ops, and small durations force equal times."""
    preds = [[] for _ in range(n_src)]
    for _ in range(groups):
        ps = sorted(rng.choice(n_src, size=int(rng.integers(2, n_src + 1)), replace=False).tolist())
        for _ in range(int(rng.integers(2, 7))):
            preds.append(ps)
    for _ in range(n_free):
        preds.append([int(rng.integers(0, n_src))])
    n = len(preds)
    perm = rng.permutation(n)  # shuffle ids (sources stay sources)
    inv = np.argsort(perm)
    succ = [[] for _ in range(n)]
    for v, ps in enumerate(preds):
        for p in ps:
            succ[perm[p]].append(int(perm[v]))
    ptr = np.zeros(n + 1, np.int64)
    ptr[1:] = np.cumsum([len(x) for x in succ])
    idx = np.array([w for x in succ for w in x], np.int32)
    res = rng.integers(0, R, n).astype(np.int32)
    prio = rng.integers(0, 4, n).astype(np.int32)
    dur = W.random_durations(n, S, 1, hi, rng)
    return ptr, idx, res, prio, dur


def test_barrier_members_interleaved(mlsim):
    """Ops sharing a predecessor set leave the ready list in the same order as
    in the oracle, also when their ready times tie with other ops."""
    rng = np.random.default_rng(404)
    for case in range(30):
        ptr, idx, res, prio, dur = barrier_case(rng, int(rng.integers(2, 6)), int(rng.integers(1, 6)),
                                                int(rng.integers(0, 12)), int(rng.integers(1, 4)),
                                                int(rng.choice([64, 130])), int(rng.choice([1, 3, 50])))
        print(f"barrier case {case} n={res.size}", flush=True)
        g = mlsim.Graph(ptr, idx, res, int(res.max()) + 1, prio=prio)
        assert g.info()["n_joins"] >= 1
        g.close()
        check_run(mlsim, ptr, idx, res, int(res.max()) + 1, dur, prio=prio)


@pytest.mark.parametrize("groups", [0, 1, 4, 8])
def test_heap_groups_in_lds(mlsim, groups, pin_variants):
    """The ready heap with some of its grandchild groups in LDS (a launch
    parameter) gives the same results as the oracle."""
    pin_variants(ev_lds_groups=groups)
    for k, S in ((4, 130), (5, 70), (2, 100)):
        w = W.make_config(k, n_scen=S)
        check_run(mlsim, w.succ_ptr, w.succ_idx, w.op_res, w.n_res, w.durations(), place=w.placement())
    rng = np.random.default_rng(77)
    for case in range(10):  # wide graphs: heaps well beyond LDS
        n, R = int(rng.integers(100, 600)), int(rng.integers(1, 5))
        ptr, idx, res, pr, dur = rand_case(rng, n, R, 0.01, bool(rng.integers(2)), False, 65, 1,
                                           int(rng.choice([3, 1000])))
        check_run(mlsim, ptr, idx, res, R, dur, prio=pr)


@pytest.mark.parametrize("groups", [0, 1, 2, 4])
def test_heap_children_in_registers(mlsim, groups, pin_variants):
    """The event kernel with the heap root's children in registers (chosen
    by the launcher when the chip is full; forced here on small and ragged
    batches), with 0-4 grandchild groups in LDS, equals the oracle: plain,
    with resource gaps and with generated durations."""
    pin_variants(ev_reg=1, ev_lds_groups=groups)
    for k, S in ((4, 130), (2, 100), (1, 1024), (3, 70)):
        w = W.make_config(k, n_scen=S if k != 1 else None)
        dur = w.durations()
        check_run(mlsim, w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur)
        gap = np.arange(w.n_res, dtype=np.int32) * 397
        g = mlsim.Graph.from_workload(w)
        mk, fin, st = g.run(dev(dur), want_finish=True, gap=gap)
        torch.cuda.synchronize()
        omk, ofin, ost = oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur, gap=gap)
        assert np.array_equal(mk.cpu().numpy(), omk) and np.array_equal(fin.cpu().numpy(), ofin)
        base = w.gen_base()
        gen = mlsim.Gen(dev(base), knob_block=29, noise=102739, seed=k)
        S2 = dur.shape[1]
        mk, fin, st = g.run_generated(gen, S2, want_finish=True)
        torch.cuda.synchronize()
        gdur = oracle.generate(base, S2, 29, 102739, k)
        omk, ofin, ost = oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, gdur)
        assert np.array_equal(mk.cpu().numpy(), omk) and np.array_equal(fin.cpu().numpy(), ofin)
        g.close()
    rng = np.random.default_rng(78)
    for case in range(12):  # random graphs with priorities, then wide ones with heaps beyond LDS
        if case < 6:
            n, R, p = int(rng.integers(1, 70)), int(rng.integers(1, 9)), float(rng.uniform(0, 0.3))
        else:
            n, R, p = int(rng.integers(100, 600)), int(rng.integers(1, 5)), 0.01
        ptr, idx, res, pr, dur = rand_case(rng, n, R, p, bool(rng.integers(2)), bool(rng.integers(2)),
                                           int(rng.choice([1, 63, 65, 130])), 1, int(rng.choice([3, 1000])))
        check_run(mlsim, ptr, idx, res, R, dur, prio=pr)


@pytest.mark.parametrize("slots", ["lds", "global"])
def test_critical_path_slots(mlsim, slots, pin_variants):
    """The critical-path sweep with its value slots in LDS or in global
    scratch, on workloads and on random graphs with sources, long predecessor
    lists (more than four, read from the list) and ops without successors;
    batch counts that leave partial batches."""
    if slots == "global":
        pin_variants(cp_global=1)
    for k, S in ((4, 130), (2, 70), (3, 200)):
        w = W.make_config(k, n_scen=S)
        check_cp(mlsim, w.succ_ptr, w.succ_idx, w.op_res, w.n_res, w.durations(), paths=(0, S - 1))
    rng = np.random.default_rng(4242)
    for case in range(12):
        n = int(rng.choice([1, 15, 16, 17, 33, 250]))
        ptr, idx, res, _ = W.random_dag(n, 3, float(rng.uniform(0.05, 0.5)), rng, with_prio=False,
                                        dup_edges=bool(rng.integers(2)))
        dur = W.random_durations(n, int(rng.choice([1, 64, 100])), 1, 1000, rng)
        check_cp(mlsim, ptr, idx, res, 3, dur, paths=(0,))


def test_single_op_and_empty(mlsim):
    check_run(mlsim, np.array([0, 0]), np.zeros(0, np.int32), np.array([0], np.int32), 1,
              np.array([[5, 1, 7]], np.int32))
    g = mlsim.Graph(np.zeros(1, np.int64), np.zeros(0, np.int32), np.zeros(0, np.int32), 1)
    mk, _, st = g.run(torch.zeros((0, 10), dtype=torch.int32, device="cuda"))
    cp, _ = g.critical_path(torch.zeros((0, 10), dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()
    assert mk.cpu().tolist() == [0] * 10 and st.cpu().tolist() == [0] * 10
    assert cp.cpu().tolist() == [0] * 10


def test_status_bits(mlsim):
    """Bad durations, bad placements and overflow match the oracle's status."""
    ptr = np.array([0, 1, 2, 2], np.int64)
    idx = np.array([1, 2], np.int32)
    res = np.zeros(3, np.int32)
    dur = np.array([[1, 0, 5, 1_500_000_000, 9, -4],
                    [1, 1, 5, 1_500_000_000, 9, 1],
                    [1, 1, 5, 1, 9, 1]], np.int32)
    place = np.array([[0, 0, 0, 0, 0, 0], [0, 1, 3, 0, 2, 0], [0, 0, 0, 0, 0, 0]], np.uint16)
    check_run(mlsim, ptr, idx, res, 1, dur)
    check_run(mlsim, ptr, idx, res, 2, dur, place=place)
    check_cp(mlsim, ptr, idx, res, 1, dur)


def test_goldens(mlsim):
    import goldens
    for g in goldens.all_goldens():
        check_run(mlsim, g["succ_ptr"], g["succ_idx"], g["op_res"], g["n_res"], g["dur"], prio=g["prio"])
        if "cp_path" in g["expect"]:
            gg = mlsim.Graph(g["succ_ptr"], g["succ_idx"], g["op_res"], g["n_res"], prio=g["prio"])
            cp, path = gg.critical_path(dev(g["dur"]), path_scen=0)
            assert cp.cpu().tolist() == g["expect"]["cp_len"]
            assert path.tolist() == g["expect"]["cp_path"]


def test_repeatable(mlsim):
    w = W.make_config(3, n_scen=500)
    dur = dev(w.durations())
    g = mlsim.Graph.from_workload(w)
    a = [t.clone() for t in g.run(dur, want_finish=True)]
    for _ in range(3):
        b = g.run(dur, want_finish=True)
        torch.cuda.synchronize()
        assert all(torch.equal(x, y) for x, y in zip(a, b))


def test_makespan_only_matches_finish_mode(mlsim):
    w = W.make_config(2, n_scen=300)
    dur = dev(w.durations())
    g = mlsim.Graph.from_workload(w)
    a, _, sa = g.run(dur, want_finish=True)
    b, _, sb = g.run(dur, want_finish=False)
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(sa, sb)


# --------------------------------------------------------------- full sizes

@pytest.mark.parametrize("k", [2, 3, 4, 5])
def test_full_size_population(mlsim, k):
    """Full scenario count in the benchmark's launch configuration: every
    scenario's makespan, status and critical path against the oracle, finish
    rows of 1024 sampled scenarios (plus the first and last)."""
    w = W.make_config(k)
    print(f"full-size {w.name} n={w.n_ops} S={w.n_scen}", flush=True)
    dur_h = w.durations()
    place_h = w.placement()
    dur = dev(dur_h)
    place = None
    if place_h is not None:
        place = torch.from_numpy(place_h.view(np.int16)).cuda().view(torch.uint16)
    g = mlsim.Graph.from_workload(w)
    mk, fin, st = g.run(dur, place=place, want_finish=True)
    cp, _ = g.critical_path(dur)
    torch.cuda.synchronize()
    mk, st, cp = mk.cpu().numpy(), st.cpu().numpy(), cp.cpu().numpy()
    print(f"  GPU done; oracle on all {w.n_scen} scenarios", flush=True)
    omk, _, ost = oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur_h, place=place_h,
                                   want_finish=False)
    print("  oracle replay done", flush=True)
    ocp, _ = oracle.critical_path(w.succ_ptr, w.succ_idx, w.n_ops, dur_h)
    assert np.array_equal(st, ost), f"status differs in {np.count_nonzero(st != ost)} scenarios"
    assert np.array_equal(mk, omk), f"makespan differs in {np.count_nonzero(mk != omk)} scenarios"
    assert np.array_equal(cp, ocp), f"critical path differs in {np.count_nonzero(cp != ocp)} scenarios"
    assert (ost == 0).all()
    rng = np.random.default_rng(k)
    scen = np.unique(np.r_[0, w.n_scen - 1, rng.choice(w.n_scen, 1024, replace=False)])
    _, ofin, _ = oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur_h[:, scen],
                                  place=None if place_h is None else place_h[:, scen])
    sel = torch.from_numpy(scen).cuda()
    assert np.array_equal(fin[:, sel].cpu().numpy(), ofin)
    assert torch.equal(fin.max(0).values.cpu(), torch.from_numpy(mk))


# ------------------------------------------------------- sweep variant (a8)

@pytest.mark.parametrize("k,S", [(1, 1024), (2, 130), (3, 200), (4, 130), (5, 70)])
def test_sweep_workload_parity(mlsim, k, S):
    w = W.make_config(k, n_scen=S if k != 1 else None)
    dur = w.durations()
    print(f"sweep workload {w.name} n={w.n_ops} S={dur.shape[1]}", flush=True)
    check_run(mlsim, w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur, place=w.placement(), algo="sweep")


def test_sweep_random_graphs(mlsim):
    rng = np.random.default_rng(99)
    for case in range(30):
        n = int(rng.integers(1, 60))
        R = int(rng.integers(1, 9))
        S = int(rng.choice([1, 63, 65, 130]))
        hi = int(rng.choice([3, 10, 1000]))
        ptr, idx, res, pr, dur = rand_case(rng, n, R, float(rng.uniform(0, 0.3)),
                                           bool(rng.integers(2)), bool(rng.integers(2)), S, 1, hi)
        place = rng.integers(0, R, size=(n, S)).astype(np.uint16) if case % 3 == 0 else None
        print(f"sweep random case {case} n={n} R={R} S={S}", flush=True)
        check_run(mlsim, ptr, idx, res, R, dur, prio=pr, place=place, algo="sweep",
                  ld_pad=int(rng.integers(0, 3)) * 5)


def test_sweep_status_and_goldens(mlsim):
    import goldens
    ptr = np.array([0, 1, 2, 2], np.int64)
    idx = np.array([1, 2], np.int32)
    res = np.zeros(3, np.int32)
    dur = np.array([[1, 0, 5, 1_500_000_000, 9, -4],
                    [1, 1, 5, 1_500_000_000, 9, 1],
                    [1, 1, 5, 1, 9, 1]], np.int32)
    place = np.array([[0, 0, 0, 0, 0, 0], [0, 1, 3, 0, 2, 0], [0, 0, 0, 0, 0, 0]], np.uint16)
    check_run(mlsim, ptr, idx, res, 1, dur, algo="sweep")
    check_run(mlsim, ptr, idx, res, 2, dur, place=place, algo="sweep")
    for g in goldens.all_goldens():
        check_run(mlsim, g["succ_ptr"], g["succ_idx"], g["op_res"], g["n_res"], g["dur"],
                  prio=g["prio"], algo="sweep")


def test_sweep_equals_event_full_bert_slice(mlsim):
    """Both algorithms agree bit for bit on a slice of every BERT strategy knob."""
    w = W.make_config(4)
    scen = np.concatenate([np.arange(k * 4096, k * 4096 + 64) for k in range(12)])
    dur_h, _ = w.columns(scen)
    dur = dev(dur_h)
    g = mlsim.Graph.from_workload(w)
    a = g.run(dur, want_finish=True, algo="event")
    b = g.run(dur, want_finish=True, algo="sweep")
    torch.cuda.synchronize()
    assert all(torch.equal(x, y) for x, y in zip(a, b))


def test_join_beyond_entry_limits(mlsim):
    """A join waiting for more predecessors than a successor entry can
    count (32768) uses the per-join table; results equal the oracle's."""
    n_src = 33000
    n = n_src + 2
    sink, tail = n_src, n_src + 1
    ptr = np.zeros(n + 1, np.int64)
    ptr[1:n_src + 1] = np.arange(1, n_src + 1)
    ptr[n_src + 1] = n_src + 1  # sink -> tail
    ptr[n_src + 2] = n_src + 1
    idx = np.r_[np.full(n_src, sink, np.int32), np.int32(tail)].astype(np.int32)
    res = (np.arange(n) % 4).astype(np.int32)
    rng = np.random.default_rng(12)
    dur = W.random_durations(n, 65, 1, 50, rng)
    print(f"join with {n_src} predecessors", flush=True)
    check_run(mlsim, ptr, idx, res, 4, dur)


def test_hip_graph_capture_replays(mlsim):
    """sim_run_batch and sim_critical_path captured in a HIP graph (through
    torch's graph capture on the current stream): each replay, with new
    durations written between replays, equals the eager calls and the
    oracle."""
    w = W.make_config(4, n_scen=192)
    G = mlsim.Graph.from_workload(w)
    rng = np.random.default_rng(5)
    durs = [w.durations()] + [np.maximum(1, w.durations() + rng.integers(-500, 500, size=(w.n_ops, 192)))
                              .astype(np.int32) for _ in range(2)]
    d = dev(durs[0])
    mk = torch.empty(192, dtype=torch.int32, device="cuda")
    st = torch.empty(192, dtype=torch.int32, device="cuda")
    fin = torch.empty((w.n_ops, 192), dtype=torch.int32, device="cuda")
    cp = torch.empty(192, dtype=torch.int32, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):  # warm up outside the capture
        G.run(d, want_finish=True, algo="event", makespan=mk, finish=fin, status=st)
        G.critical_path(d, cp_len=cp)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        G.run(d, want_finish=True, algo="event", makespan=mk, finish=fin, status=st)
        G.critical_path(d, cp_len=cp)
    for rep in range(3):
        dh = durs[rep % len(durs)]
        d.copy_(torch.from_numpy(dh))  # eager work between replays
        graph.replay()
        torch.cuda.synchronize()
        emk, efin, est = G.run(d, want_finish=True, algo="event")
        ecp, _ = G.critical_path(d)
        torch.cuda.synchronize()
        assert torch.equal(mk, emk) and torch.equal(fin, efin) and torch.equal(st, est) and torch.equal(cp, ecp)
        omk, _, _ = oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dh, want_finish=False)
        assert np.array_equal(mk.cpu().numpy(), omk), f"replay {rep}"
    G.close()


# ------------------------------------------------ pinned kernel variants

def _variant_cases(mlsim):
    for k, S in ((4, 130), (2, 100), (5, 70), (1, 1024), (3, 70)):
        w = W.make_config(k, n_scen=S if k != 1 else None)
        check_run(mlsim, w.succ_ptr, w.succ_idx, w.op_res, w.n_res, w.durations(), place=w.placement())
    rng = np.random.default_rng(4077)
    for case in range(12):
        if case < 6:
            ptr, idx, res, prio, dur = barrier_case(rng, int(rng.integers(2, 6)), int(rng.integers(1, 6)),
                                                    int(rng.integers(0, 12)), int(rng.integers(1, 4)),
                                                    int(rng.choice([64, 130])), int(rng.choice([1, 3, 50])))
            R = int(res.max()) + 1
        else:
            n, R = int(rng.integers(100, 400)), int(rng.integers(1, 5))
            ptr, idx, res, prio, dur = rand_case(rng, n, R, 0.01, bool(rng.integers(2)), False, 65, 1,
                                                 int(rng.choice([3, 1000])))
        check_run(mlsim, ptr, idx, res, R, dur, prio=prio)


def test_resource_times_in_global_memory(mlsim, pin_variants):
    """The event kernel with its resource times (and the attribution's
    last-op table) in global scratch instead of LDS equals the oracle."""
    pin_variants(rf_global=1)
    _variant_cases(mlsim)
    w = W.make_config(2, n_scen=100)
    dur = w.durations()
    g = mlsim.Graph.from_workload(w)
    gap = np.arange(w.n_res, dtype=np.int32) * 311
    delay = (np.arange(w.n_res, dtype=np.int32) % 3) * 1000
    mk, fin, _ = g.run(dev(dur), want_finish=True, gap=gap, delay=delay)
    h = g.attribute(dev(dur))
    torch.cuda.synchronize()
    omk, ofin, _ = oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur, gap=gap, delay=delay)
    assert np.array_equal(mk.cpu().numpy(), omk) and np.array_equal(fin.cpu().numpy(), ofin)
    amk, _, _ = oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur)
    assert np.array_equal(h["makespan"].cpu().numpy(), amk)


@pytest.mark.parametrize("cap", [1, 3])
def test_event_grid_cap(mlsim, cap, pin_variants):
    """A persistent grid of only 1 or 3 blocks walks every tile in turn."""
    pin_variants(ev_blocks_cap=cap)
    w = W.make_config(2, n_scen=64 * 7 + 5)
    check_run(mlsim, w.succ_ptr, w.succ_idx, w.op_res, w.n_res, w.durations())
    w = W.make_config(5, n_scen=64 * 4 + 1)
    check_run(mlsim, w.succ_ptr, w.succ_idx, w.op_res, w.n_res, w.durations(), place=w.placement())


# --------------------------------------------------- streams and the boundary

def test_two_streams_share_one_graph(mlsim):
    """Overlapping calls on two streams with one graph (replays with
    different resource gaps, whose tables live in the calls' scratch sets,
    critical paths and plain replays) each equal the oracle."""
    w = W.make_config(2, n_scen=640)
    g = mlsim.Graph.from_workload(w)
    dh = [w.durations(), np.maximum(1, w.durations() // 2 + 7).astype(np.int32)]
    d = [dev(x) for x in dh]
    gaps = [np.full(w.n_res, 1500, np.int32), np.arange(w.n_res, dtype=np.int32) * 37]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    out = [[], []]
    for rep in range(3):  # issue everything before waiting for anything
        for i, s in enumerate(streams):
            with torch.cuda.stream(s):
                out[i].append(g.run(d[i], want_finish=True, gap=gaps[i]))
                out[i].append(g.critical_path(d[i])[0])
                out[i].append(g.run(d[i], want_finish=False))
    torch.cuda.synchronize()
    for i in range(2):
        omk, ofin, ost = oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dh[i], gap=gaps[i])
        pmk, _, _ = oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dh[i], want_finish=False)
        ocp, _ = oracle.critical_path(w.succ_ptr, w.succ_idx, w.n_ops, dh[i])
        for rep in range(3):
            mk, fin, st = out[i][3 * rep]
            assert np.array_equal(mk.cpu().numpy(), omk), (i, rep)
            assert np.array_equal(fin.cpu().numpy(), ofin), (i, rep)
            assert np.array_equal(out[i][3 * rep + 1].cpu().numpy(), ocp), (i, rep)
            assert np.array_equal(out[i][3 * rep + 2][0].cpu().numpy(), pmk), (i, rep)
    g.close()


def test_two_streams_sweep_beside_event(mlsim):
    """The sweep variant keeps its state in scratch sets of its own: sweeps
    and event replays issued on two streams at once, over one graph, each
    equal the oracle."""
    w = W.make_config(3, n_scen=640)
    g = mlsim.Graph.from_workload(w)
    dh = [w.durations(), np.maximum(1, w.durations() // 3 + 11).astype(np.int32)]
    d = [dev(x) for x in dh]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    out = [[], []]
    for rep in range(2):  # issue everything before waiting for anything
        for i, s in enumerate(streams):
            with torch.cuda.stream(s):
                out[i].append(g.run(d[i], algo="sweep", want_finish=True))
                out[i].append(g.run(d[1 - i], algo="event", want_finish=True))
    torch.cuda.synchronize()
    ref = [oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, x, prio=w.prio) for x in dh]
    for i in range(2):
        for rep in range(2):
            for k, src in ((0, i), (1, 1 - i)):
                mk, fin, st = out[i][2 * rep + k]
                omk, ofin, ost = ref[src]
                assert np.array_equal(mk.cpu().numpy(), omk), (i, rep, k)
                assert np.array_equal(st.cpu().numpy(), ost), (i, rep, k)
                assert np.array_equal(fin.cpu().numpy(), ofin), (i, rep, k)
    g.close()


def test_binding_rejects_bad_arrays(mlsim):
    """Output and input arrays that would let a kernel read or write out of
    bounds are rejected before the call."""
    w = W.make_config(1, n_scen=100)
    g = mlsim.Graph.from_workload(w)
    d = dev(w.durations())
    with pytest.raises(ValueError):
        g.run(d, makespan=torch.empty(99, dtype=torch.int32, device="cuda"))
    with pytest.raises(ValueError):
        g.run(d, status=torch.empty(100, dtype=torch.int64, device="cuda"))
    with pytest.raises(TypeError):
        g.run(d, makespan=torch.empty(100, dtype=torch.int32))
    with pytest.raises(ValueError):
        g.run(d, finish=torch.empty((w.n_ops, 50), dtype=torch.int32, device="cuda"))
    with pytest.raises(ValueError):  # one row expanded over every op: rows overlap
        g.run(d[:1].expand(w.n_ops, 100))
    with pytest.raises(ValueError):
        g.critical_path(d, cp_len=torch.empty(10, dtype=torch.int32, device="cuda"))
    big = torch.empty(200, dtype=torch.int32, device="cuda")  # longer outputs are fine
    mk, _, _ = g.run(d, makespan=big)
    torch.cuda.synchronize()
    omk, _, _ = oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, w.durations(), want_finish=False)
    assert np.array_equal(big[:100].cpu().numpy(), omk)
    g.close()


def test_threads_share_one_graph(mlsim):
    """Four host threads, each with its own stream, call one graph at once
    (the calls take scratch sets under the graph's lock); every result
    equals the oracle."""
    import threading
    w = W.make_config(3, n_scen=256)
    g = mlsim.Graph.from_workload(w)
    dh = [np.maximum(1, w.durations() // (i + 1)).astype(np.int32) for i in range(4)]
    d = [dev(x) for x in dh]
    torch.cuda.synchronize()
    out, errors = [None] * 4, []

    def work(i):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                res = []
                for _ in range(5):
                    res.append(g.run(d[i], want_finish=True, gap=np.full(w.n_res, 100 * i, np.int32)))
                    res.append(g.critical_path(d[i])[0])
            s.synchronize()
            out[i] = res
        except Exception as e:  # reported below
            errors.append(e)

    ts = [threading.Thread(target=work, args=(i,)) for i in range(4)]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for i in range(4):
        omk, ofin, _ = oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dh[i],
                                        gap=np.full(w.n_res, 100 * i, np.int32))
        ocp, _ = oracle.critical_path(w.succ_ptr, w.succ_idx, w.n_ops, dh[i])
        for rep in range(5):
            mk, fin, _ = out[i][2 * rep]
            assert np.array_equal(mk.cpu().numpy(), omk) and np.array_equal(fin.cpu().numpy(), ofin), (i, rep)
            assert np.array_equal(out[i][2 * rep + 1].cpu().numpy(), ocp), (i, rep)
    g.close()
