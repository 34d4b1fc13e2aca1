"""The replay entry point that allocates nothing (sim_run_batch_noalloc).

Its scratch is one fixed array in the library's static device memory; every
call goes through the C ABI here and is compared bit for bit with
sim_run_batch on the same inputs (and with the oracle), on two calls in a
row with the second smaller, across graphs whose scratch layouts differ,
with placement, with more tiles than the array holds blocks, and for a
graph whose per-block scratch exceeds the array.
"""
import ctypes
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


def noalloc(mlsim, g, dur, place=None, want_finish=True):
    """sim_run_batch_noalloc through the C ABI; outputs as device tensors."""
    n, S = dur.shape
    mk = torch.full((S,), -7, dtype=torch.int32, device="cuda")
    st = torch.full((S,), -7, dtype=torch.int32, device="cuda")
    fin = torch.full((n, S), -7, dtype=torch.int32, device="cuda") if want_finish else None
    stream = torch.cuda.current_stream().cuda_stream
    rc = mlsim.lib().sim_run_batch_noalloc(
        g._h, S, dur.data_ptr(), dur.stride(0), None if place is None else place.data_ptr(),
        0 if place is None else place.stride(0), mk.data_ptr(), None if fin is None else fin.data_ptr(),
        S if fin is not None else 0, st.data_ptr(), 0, ctypes.c_void_p(stream))
    assert rc == 0, mlsim.lib().sim_strerror(rc)
    return mk, fin, st


def check(mlsim, w, S, place_on=True):
    dur_h, place_h = w.columns(np.arange(S))
    if not place_on:
        place_h = None
    d = dev(dur_h)
    p = None if place_h is None else torch.from_numpy(place_h.view(np.int16)).cuda().view(torch.uint16)
    g = mlsim.Graph.from_workload(w)
    print(f"noalloc {w.name} n={w.n_ops} S={S} place={p is not None}", flush=True)
    mk, fin, st = noalloc(mlsim, g, d, p)
    rmk, rfin, rst = g.run(d, place=p, want_finish=True, algo="event")
    torch.cuda.synchronize()
    assert torch.equal(mk, rmk) and torch.equal(st, rst) and torch.equal(fin, rfin)
    omk, _, ost = oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur_h, place=place_h,
                                   want_finish=False)
    assert np.array_equal(mk.cpu().numpy(), omk) and np.array_equal(st.cpu().numpy(), ost)
    return g


def test_noalloc_two_calls_second_smaller(mlsim):
    w = W.make_config(4, n_scen=4096)
    g = check(mlsim, w, 1000)      # ragged: 16 tiles, the last one partial
    check(mlsim, w, 70)            # smaller, same graph
    g.close()


def test_noalloc_other_layouts_between_calls(mlsim):
    """Graphs with other heap and join layouts use the same array in turn."""
    for k, S in ((2, 300), (5, 130), (3, 65), (1, 1024), (4, 64)):
        check(mlsim, W.make_config(k, n_scen=max(S, 64) if k != 1 else None), S).close()


def test_noalloc_more_tiles_than_blocks(mlsim):
    """A wide graph whose heap bound leaves room for few blocks in the
    array: the persistent grid takes several rounds of tiles."""
    rng = np.random.default_rng(31)
    n, R = 12000, 3
    ptr, idx, res, _ = W.random_dag(n, R, 0.00002, rng, with_prio=False)
    dur_h = W.random_durations(n, 64 * 40 + 3, 1, 1000, rng)
    g = mlsim.Graph(ptr, idx, res, R)
    d = dev(dur_h)
    for S in (64 * 40 + 3, 64 * 3 + 1):
        mk, fin, st = noalloc(mlsim, g, d[:, :S])
        rmk, rfin, rst = g.run(d[:, :S], want_finish=True, algo="event")
        torch.cuda.synchronize()
        assert torch.equal(mk, rmk) and torch.equal(fin, rfin) and torch.equal(st, rst), S
    omk, _, _ = oracle.run_batch(ptr, idx, res, R, dur_h[:, :64 * 3 + 1], want_finish=False)
    assert np.array_equal(mk.cpu().numpy(), omk)
    g.close()


def test_noalloc_rejects_scratch_beyond_the_array(mlsim):
    """270000 ops that are all ready at once need more heap per block than
    the array holds: the call returns SIM_E_LIMIT before any launch."""
    n = 270000
    g = mlsim.Graph(np.zeros(n + 1, np.int64), np.zeros(0, np.int32), np.zeros(n, np.int32), 1)
    d = torch.ones((n, 1), dtype=torch.int32, device="cuda")
    mk = torch.empty(1, dtype=torch.int32, device="cuda")
    rc = mlsim.lib().sim_run_batch_noalloc(g._h, 1, d.data_ptr(), 1, None, 0, mk.data_ptr(), None, 0, None, 0,
                                           ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == mlsim.SIM_E_LIMIT
    g.close()
