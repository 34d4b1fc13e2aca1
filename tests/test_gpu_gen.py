"""GPU parity of on-device scenario generation (knob grid x Philox noise).

The library generates durations inside its kernels (sim_generate,
sim_run_generated, sim_critical_path_generated); the oracle generates the
same durations on the CPU from the same definition (oracle_generate) and
replays them.  Every comparison is element by element and bit-exact.
"""
import os

import numpy as np
import pytest

import oracle
from paper_2002_06790_amd import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

SIGMA1 = 102739  # 1 % relative noise


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


def gen_of(mlsim, base, knob_block, noise, seed, scen0):
    return mlsim.Gen(dev(base), knob_block=knob_block, noise=noise, seed=seed, scen0=scen0)


CASES = [  # (workload, scenarios, knob block, scen0, seed)
    (1, 1024, 1, 0, 1),
    (2, 200, 1, 2**32 - 100, 2),  # the counter's high word changes inside the batch
    (3, 333, 1, 12345, 2**64 - 1),
    (4, 200, 37, 4096 * 11 - 50, 4),  # knobs change inside a wavefront
    (5, 130, 1, 0, 5),
]


@pytest.mark.parametrize("k,S,kb,scen0,seed", CASES)
def test_generate_matches_oracle(mlsim, k, S, kb, scen0, seed):
    w = W.make_config(k, n_scen=64)
    base = w.gen_base()
    print(f"generate {w.name} knobs={base.shape[0]} S={S} scen0={scen0}", flush=True)
    g = gen_of(mlsim, base, kb, SIGMA1, seed, scen0)
    out = torch.full((w.n_ops, S + 3), -7, dtype=torch.int32, device="cuda")
    mlsim.generate(g, S, out=out[:, :S])
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    want = oracle.generate(base, S, kb, SIGMA1, seed, scen0=scen0)
    assert np.array_equal(got[:, :S], want)
    assert (got[:, S:] == -7).all(), "wrote past n_scen"


@pytest.mark.parametrize("k,S,kb,scen0,seed", CASES)
def test_run_generated_matches_oracle(mlsim, k, S, kb, scen0, seed):
    w = W.make_config(k, n_scen=64)
    base = w.gen_base()
    print(f"run_generated {w.name} S={S} scen0={scen0}", flush=True)
    G = mlsim.Graph.from_workload(w)
    g = gen_of(mlsim, base, kb, SIGMA1, seed, scen0)
    mk, fin, st = G.run_generated(g, S, want_finish=True)
    cp, _ = G.critical_path_generated(g, S)
    torch.cuda.synchronize()
    dur = oracle.generate(base, S, kb, SIGMA1, seed, scen0=scen0)
    omk, ofin, ost = oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur, prio=w.prio)
    assert np.array_equal(st.cpu().numpy(), ost)
    assert (ost == 0).all()
    assert np.array_equal(mk.cpu().numpy(), omk)
    assert np.array_equal(fin.cpu().numpy(), ofin)
    ocp, _ = oracle.critical_path(w.succ_ptr, w.succ_idx, w.n_ops, dur)
    assert np.array_equal(cp.cpu().numpy(), ocp)
    for s in (0, S - 1):
        _, path = G.critical_path_generated(g, S, path_scen=s)
        _, opath = oracle.critical_path(w.succ_ptr, w.succ_idx, w.n_ops, dur, path_scen=s)
        assert np.array_equal(path, opath), f"path of scenario {s}"
    G.close()


def test_generated_equals_explicit_durations(mlsim):
    """Generating in the kernel and replaying a written-out matrix agree."""
    w = W.make_config(4, n_scen=64)
    base = w.gen_base()
    S = 8192 + 77
    G = mlsim.Graph.from_workload(w)
    g = gen_of(mlsim, base, 4096, SIGMA1, 77, 4096 * 3)
    dur = mlsim.generate(g, S)
    mk, fin, st = G.run(dur, want_finish=True, algo="event")
    gmk, gfin, gst = G.run_generated(g, S, want_finish=True)
    cp, _ = G.critical_path(dur)
    gcp, _ = G.critical_path_generated(g, S)
    torch.cuda.synchronize()
    assert torch.equal(st, gst) and int(st.abs().sum()) == 0
    assert torch.equal(mk, gmk)
    assert torch.equal(fin, gfin)
    assert torch.equal(cp, gcp)
    G.close()


def test_invalid_base_and_zero_noise(mlsim):
    """Bases outside [1, 2^24] flag exactly the scenarios whose knob holds
    them; without noise the durations are the bases."""
    w = W.make_config(1)
    base = np.stack([w.gen_base()[0]] * 3)
    base[1, 5] = 0
    base[2, 7] = 2**24 + 1
    S = 300
    G = mlsim.Graph.from_workload(w)
    for noise in (0, SIGMA1):
        g = gen_of(mlsim, base, 5, noise, 9, 0)
        mk, fin, st = G.run_generated(g, S, want_finish=True)
        cp, _ = G.critical_path_generated(g, S)
        torch.cuda.synchronize()
        dur = oracle.generate(base, S, 5, noise, 9)
        if noise == 0:
            b = base[(np.arange(S) // 5) % 3].T
            assert np.array_equal(dur, np.where((b >= 1) & (b <= 2**24), b, 0))
        omk, ofin, ost = oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur)
        ocp, _ = oracle.critical_path(w.succ_ptr, w.succ_idx, w.n_ops, dur)
        st = st.cpu().numpy()
        assert np.array_equal(st, ost)
        assert set(np.nonzero(ost)[0] // 5 % 3) == {1, 2}
        assert np.array_equal(mk.cpu().numpy(), omk)
        ok = ost == 0
        assert np.array_equal(fin.cpu().numpy()[:, ok], ofin[:, ok])
        assert np.array_equal(cp.cpu().numpy(), ocp)
    G.close()


def test_bert_full_size_sampled(mlsim):
    """BERT at its full 262144 scenarios (the benchmark's launch shape):
    sampled scenarios equal the oracle's replay of the same generated
    durations."""
    w = W.make_config(4)
    base = w.gen_base()
    S = w.n_scen
    G = mlsim.Graph.from_workload(w)
    g = gen_of(mlsim, base, w.knob_block, SIGMA1, 2002067904, 0)
    mk, _, st = G.run_generated(g, S)
    cp, _ = G.critical_path_generated(g, S)
    torch.cuda.synchronize()
    mk, st, cp = mk.cpu().numpy(), st.cpu().numpy(), cp.cpu().numpy()
    assert (st == 0).all()
    rng = np.random.default_rng(3)
    sample = np.unique(np.concatenate([[0, 4095, 4096, S - 1], rng.integers(0, S, 44)]))
    for s in sample:
        dur = oracle.generate(base, 1, w.knob_block, SIGMA1, 2002067904, scen0=int(s))
        omk, _, _ = oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur, want_finish=False)
        ocp, _ = oracle.critical_path(w.succ_ptr, w.succ_idx, w.n_ops, dur)
        assert mk[s] == omk[0], f"scenario {s}"
        assert cp[s] == ocp[0], f"scenario {s}"
    # properties at every scenario: the longest path bounds the iteration
    assert (cp <= mk).all()
    G.close()


def test_empty_and_tiny(mlsim):
    w = W.make_config(1)
    base = w.gen_base()
    G = mlsim.Graph.from_workload(w)
    g = gen_of(mlsim, base, 1, SIGMA1, 1, 0)
    mk, _, st = G.run_generated(g, 0)
    assert mk.numel() == 0
    mk, fin, st = G.run_generated(g, 1, want_finish=True)
    torch.cuda.synchronize()
    dur = oracle.generate(base, 1, 1, SIGMA1, 1)
    omk, ofin, _ = oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur)
    assert mk.cpu().numpy()[0] == omk[0]
    assert np.array_equal(fin.cpu().numpy(), ofin)
    with pytest.raises(mlsim.SimError):
        G.run_generated(g, 4, algo="sweep")
    G.close()


@pytest.mark.parametrize("k", [1, 2, 4])
def test_static_replay_generated(mlsim, k):
    """The static-order replay on generated durations equals the oracle's
    static-order replay of the oracle's generated durations."""
    w = W.make_config(k, n_scen=64)
    base = w.gen_base()
    S = 150
    G = mlsim.Graph.from_workload(w)
    order = np.arange(w.n_ops, dtype=np.int32)  # op ids are emitted in topological order
    sr = G.static_order(order)
    g = gen_of(mlsim, base, 7, SIGMA1, 11, 3)
    mk, fin, st = sr.run_generated(g, S, want_finish=True)
    mk0, _, st0 = sr.run_generated(g, S)
    torch.cuda.synchronize()
    dur = oracle.generate(base, S, 7, SIGMA1, 11, scen0=3)
    omk, ofin, ost = oracle.static_run(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, order, dur)
    assert np.array_equal(st.cpu().numpy(), ost) and (ost == 0).all()
    assert np.array_equal(mk.cpu().numpy(), omk) and np.array_equal(mk0.cpu().numpy(), omk)
    assert np.array_equal(fin.cpu().numpy(), ofin)
    sr.close()
    G.close()
