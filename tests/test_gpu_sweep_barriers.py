"""GPU parity of the max-plus sweep on tables with barrier records.

When several ops share one predecessor set, the sweep table may stand the set
for one barrier record (the max over the set, duration 0) that those ops read
instead of the whole set.  The graphs here are built so that the barrier table
needs fewer live values than any table without it (m sources that all feed k
joins, each join followed by a chain), so the library picks it.  The critical
path, the static-order replay (every op on its own resource, so the replay
table is the same DAG) and the generated-duration sweep are compared with the
oracle, including the status cases: a bad duration of op 0 (whose row a
barrier reads), a path of exactly INT32_MAX, one just above it, and sums that
would wrap 32 bits.
"""
import os

import numpy as np
import pytest

import oracle
from paper_2002_06790_amd import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

I32MAX = 2**31 - 1


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


def fan_graph(m, k, chain):
    """Sources 0..m-1 all feed joins m..m+k-1; join j starts a chain of
    `chain` ops.  Returns successor CSR and n."""
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
    ptr[1:] = np.cumsum([len(s) for s in succ])
    idx = np.array([w for s in succ for w in s], np.int32)
    return ptr, idx, n


def status_columns(n, m, k, chain):
    """Columns for the status cases of fan_graph(m, k, chain): the longest
    path is source + join + chain ops."""
    cols = []

    def col(src0=1, other=1):
        c = np.full(n, other, np.int64)
        c[0] = src0
        return c

    c = col(); c[0] = 0; cols.append(c)                 # op 0 (read by the barrier) bad
    c = col(); c[0] = -7; cols.append(c)                # negative
    c = col(); c[m + k] = 0; cols.append(c)             # a chain op bad
    base = I32MAX - (1 + chain)                         # source + join + chain = INT32_MAX exactly
    cols.append(col(src0=base))
    cols.append(col(src0=base + 1))                     # one above: overflow
    cols.append(np.full(n, I32MAX, np.int64))           # every sum would wrap
    cols.append(np.full(n, 2**30, np.int64))            # source + join = 2^31: overflow before any wrap
    return np.stack(cols, 1).astype(np.int32)


CASES = [(6, 6, 2), (5, 4, 1), (3, 3, 1), (8, 3, 2)]  # barrier of > 4 and of <= 4 predecessors


@pytest.mark.parametrize("m,k,chain", CASES)
@pytest.mark.parametrize("slots", ["lds", "global"])
def test_critical_path_barrier_table(mlsim, m, k, chain, slots, pin_variants):
    if slots == "global":
        pin_variants(cp_global=1)
    ptr, idx, n = fan_graph(m, k, chain)
    rng = np.random.default_rng(1000 * m + 10 * k + chain)
    dur = np.concatenate([W.random_durations(n, 190, 1, 1000, rng), status_columns(n, m, k, chain)], 1)
    S = dur.shape[1]
    print(f"fan graph m={m} k={k} chain={chain} slots={slots} S={S}", flush=True)
    g = mlsim.Graph(ptr, idx, np.zeros(n, np.int32), 1)
    d = dev(dur)
    cp, _ = g.critical_path(d)
    torch.cuda.synchronize()
    ocp, _ = oracle.critical_path(ptr, idx, n, dur)
    assert np.array_equal(cp.cpu().numpy(), ocp)
    assert (ocp[190:] == -1).sum() == 6 and ocp[190 + 3] == I32MAX
    for s in (0, 7, 189, 190, 193):
        _, path = g.critical_path(d, path_scen=s)
        _, opath = oracle.critical_path(ptr, idx, n, dur, path_scen=s)
        assert np.array_equal(path, opath), f"path of scenario {s}"
    g.close()


@pytest.mark.parametrize("m,k,chain", CASES)
def test_static_replay_barrier_table(mlsim, m, k, chain):
    """Every op on its own resource: the replay table is the DAG's, with the
    barrier; finish rows of unflagged scenarios and all statuses match."""
    ptr, idx, n = fan_graph(m, k, chain)
    rng = np.random.default_rng(77 + m)
    dur = np.concatenate([W.random_durations(n, 120, 1, 1000, rng), status_columns(n, m, k, chain)], 1)
    res = np.arange(n, dtype=np.int32)
    order = np.arange(n, dtype=np.int32)
    g = mlsim.Graph(ptr, idx, res, n)
    st_obj = g.static_order(order)
    mk, fin, st = st_obj.run(dev(dur), want_finish=True)
    torch.cuda.synchronize()
    omk, ofin, ost = oracle.static_run(ptr, idx, res, n, order, dur)
    assert np.array_equal(st.cpu().numpy(), ost)
    assert np.array_equal(mk.cpu().numpy(), omk)
    ok = ost == 0
    assert np.array_equal(fin.cpu().numpy()[:, ok], ofin[:, ok])
    assert (ost[120:] != 0).sum() == 6
    # with unlimited resources the static replay is the critical path
    ocp, _ = oracle.critical_path(ptr, idx, n, dur)
    assert np.array_equal(omk, ocp)
    st_obj.close()
    g.close()


def test_generated_barrier_table(mlsim):
    """Generated durations: an invalid base of op 0 in one knob flags exactly
    that knob's scenarios, also through the barrier that reads op 0's row."""
    m, k, chain = 6, 6, 2
    ptr, idx, n = fan_graph(m, k, chain)
    rng = np.random.default_rng(5)
    base = rng.integers(1000, 5000, size=(3, n)).astype(np.int32)
    base[1, 0] = 0
    S, kb = 300, 7
    g = mlsim.Graph(ptr, idx, np.zeros(n, np.int32), 1)
    gen = mlsim.Gen(dev(base), knob_block=kb, noise=102739, seed=11, scen0=0)
    cp, _ = g.critical_path_generated(gen, S)
    torch.cuda.synchronize()
    dur = oracle.generate(base, S, kb, 102739, 11)
    ocp, _ = oracle.critical_path(ptr, idx, n, dur)
    assert np.array_equal(cp.cpu().numpy(), ocp)
    assert set(np.nonzero(ocp < 0)[0] // kb % 3) == {1}
    g.close()
