"""The seeded workload generators: shapes, determinism, value ranges, headroom."""
import numpy as np
import pytest

import oracle
from paper_2002_06790_amd import workloads as W

EXPECT = {  # name, n_ops, n_res, n_scen (exact counts of the generators)
    1: ("tiny-dp-mlp", 42, 3, 1024),
    2: ("resnet50-ps", 4574, 17, 65536),
    3: ("inception-v3-ring", 1104, 8, 65536),
    4: ("bert-large-ps", 6624, 48, 262144),
    5: ("random-layered", 20000, 64, 16384),
}


@pytest.mark.parametrize("k", sorted(EXPECT))
def test_shapes_and_acyclic(k):
    name, n, R, S = EXPECT[k]
    w = W.make_config(k)
    assert (w.name, w.n_ops, w.n_res, w.n_scen) == (name, n, R, S)
    assert w.succ_ptr.shape == (n + 1,) and w.succ_ptr[0] == 0
    assert (np.diff(w.succ_ptr) >= 0).all()
    assert w.succ_idx.dtype == np.int32 and w.op_res.dtype == np.int32
    assert ((w.op_res >= 0) & (w.op_res < R)).all()
    # ids are emitted in topological order, so every edge points forward
    src = np.repeat(np.arange(n), np.diff(w.succ_ptr))
    assert (w.succ_idx > src).all()
    # every resource is used
    assert np.unique(w.op_res).size == R or w.has_place


def test_tiny_mlp_edges():
    w = W.make_config(1)
    assert w.n_edges == 46


@pytest.mark.parametrize("k", sorted(EXPECT))
def test_durations_deterministic_and_positive(k):
    w = W.make_config(k, n_scen=300)
    a = w.durations(threads=1)
    b = W.make_config(k, n_scen=300).durations(threads=3)
    assert a.dtype == np.int32 and a.shape == (w.n_ops, 300)
    assert (a == b).all() and (a >= 1).all()
    sel = np.array([0, 7, 299])
    d, p = w.columns(sel)
    assert (d == a[:, sel]).all()
    if w.has_place:
        pa = w.placement()
        assert (p == pa[:, sel]).all() and pa.max() < w.n_res
    # the 1 % perturbation: columns differ, but only slightly (apart from C5)
    if k in (1, 2, 3):
        rel = np.abs(a[:, 1].astype(float) / a[:, 0] - 1)
        assert 0 < np.median(rel) < 0.03


def test_blocks_span_scenarios():
    w = W.make_config(4, n_scen=W.BLOCK + 10)
    d = w.durations()
    d2, _ = w.columns(np.array([W.BLOCK - 1, W.BLOCK, W.BLOCK + 9]))
    assert (d2 == d[:, [W.BLOCK - 1, W.BLOCK, W.BLOCK + 9]]).all()


def test_bert_knob_headroom():
    """The heaviest strategy knob (batch x4, 10 GB/s) stays well below 2^31 ns."""
    w = W.make_config(4)
    bf, bw = W.BERT_KNOBS[9]
    assert (bf, bw) == (4.0, 10.0)
    scen = np.array([9 * 4096, 9 * 4096 + 1])
    dur, _ = w.columns(scen)
    mk, _, st = oracle.run_batch(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, dur, want_finish=False)
    assert (st == 0).all()
    assert mk.max() < 2**31 // 3


def test_link_resources_carry_transfers_only():
    """The resources offered for bandwidth sharing exist, are distinct and
    run ops; every workload keeps some compute resource outside them."""
    for k in (1, 2, 3, 4, 5):
        w = W.make_config(k, n_scen=64)
        links = W.link_resources(w)
        assert np.all((links >= 0) & (links < w.n_res)) and np.unique(links).size == links.size
        used = np.bincount(w.op_res, minlength=w.n_res)
        assert np.all(used[links] > 0)
        assert links.size < w.n_res  # some resource computes
