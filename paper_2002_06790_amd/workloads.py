"""Seeded synthetic workloads for the batched dataflow replay.

A workload is one training iteration written as a dataflow graph: ops are
nodes, data and synchronisation are edges, and every op is pinned to one
resource (a device stream or a communication link), as in the paper's
"Dataflow based simulation" paragraph (Sec. 2).  Each of ``n_scen``
scenarios gives every op an integer-nanosecond duration; durations are laid
out op-major x scenario (``dur[v, s]``) so that one op's durations for
consecutive scenarios are contiguous.

The paper's own inputs (TensorFlow graphs of VGG/ResNet with per-op profiles
measured on V100, Table 2) are not available.  These graphs stand in for them:
their shapes follow the public model architectures (ResNet-50,
Inception-v3, BERT-large) and parallelisation schemes the paper names
(parameter server, all-reduce; Sec. 1), and durations are drawn from seeded
distributions with a 1 % lognormal per-op perturbation (the paper reports
op-profile standard errors below 1 % of the mean, Sec. 3).

This module holds structure and random numbers only: nothing here orders,
schedules or sums durations along the graph.  It is the one module shared by
the CPU oracle's tests and the GPU path's tests and benchmark.
"""
from __future__ import annotations

import concurrent.futures as _cf
import dataclasses
import os
from typing import Callable, Optional

import numpy as np

#: scenarios per random-number block; durations of block ``b`` come from their
#: own seeded stream, so any subset of scenarios can be regenerated alone.
BLOCK = 4096

_SEED_BASE = 2002067900


def _rng(seed: int, *key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=key)))


def _log_uniform(rng: np.random.Generator, lo: float, hi: float, size) -> np.ndarray:
    return np.exp(rng.uniform(np.log(lo), np.log(hi), size=size))


def _to_ns(x: np.ndarray) -> np.ndarray:
    """float ns -> int32 ns: round half to even, then clamp to at least 1 ns."""
    np.rint(x, out=x)
    np.maximum(x, 1.0, out=x)
    if x.size and float(x.max()) > 2**31 - 1:
        raise OverflowError("generated duration exceeds int32")
    return x.astype(np.int32)


@dataclasses.dataclass
class Workload:
    """Graph in successor-CSR form plus a seeded duration (and placement) source."""

    name: str
    n_ops: int
    n_res: int
    succ_ptr: np.ndarray  # int64 [n_ops + 1]
    succ_idx: np.ndarray  # int32 [succ_ptr[-1]]
    op_res: np.ndarray  # int32 [n_ops]
    n_scen: int
    seed: int
    prio: Optional[np.ndarray] = None  # int32 [n_ops] or None (priority = op id)
    # block -> float64 [n_ops, BLOCK] of un-rounded ns durations
    _dur_block: Callable[[int], np.ndarray] = dataclasses.field(default=None, repr=False)
    # block -> uint16 [n_ops, BLOCK] per-scenario resource of each op, or None
    _place_block: Optional[Callable[[int], np.ndarray]] = dataclasses.field(default=None, repr=False)
    info: dict = dataclasses.field(default_factory=dict)
    # float64 [n_knobs, n_ops] un-rounded base ns per strategy knob, and the
    # number of consecutive scenarios that share a knob (on-device generation)
    _gen_base: Optional[np.ndarray] = dataclasses.field(default=None, repr=False)
    knob_block: int = 1

    @property
    def n_edges(self) -> int:
        return int(self.succ_ptr[-1])

    @property
    def has_place(self) -> bool:
        return self._place_block is not None

    # -- durations -----------------------------------------------------------
    def _block_cols(self, b: int) -> int:
        return min(BLOCK, self.n_scen - b * BLOCK)

    def dur_block(self, b: int) -> np.ndarray:
        """int32 [n_ops, cols] durations of scenarios [b*BLOCK, b*BLOCK+cols)."""
        cols = self._block_cols(b)
        x = self._dur_block(b)[:, :cols]
        return _to_ns(np.ascontiguousarray(x))

    def place_block(self, b: int) -> Optional[np.ndarray]:
        if self._place_block is None:
            return None
        cols = self._block_cols(b)
        return np.ascontiguousarray(self._place_block(b)[:, :cols])

    def _fill(self, fn, out: np.ndarray, threads: Optional[int]) -> np.ndarray:
        nblk = (self.n_scen + BLOCK - 1) // BLOCK

        def one(b):
            blk = fn(b)
            out[:, b * BLOCK: b * BLOCK + blk.shape[1]] = blk

        threads = threads or min(16, len(os.sched_getaffinity(0)))
        if nblk == 1 or threads <= 1:
            for b in range(nblk):
                one(b)
        else:
            with _cf.ThreadPoolExecutor(threads) as ex:
                list(ex.map(one, range(nblk)))
        return out

    def durations(self, threads: Optional[int] = None) -> np.ndarray:
        """All durations, int32 [n_ops, n_scen] (op-major x scenario)."""
        out = np.empty((self.n_ops, self.n_scen), np.int32)
        return self._fill(self.dur_block, out, threads)

    def placement(self, threads: Optional[int] = None) -> Optional[np.ndarray]:
        """All placements, uint16 [n_ops, n_scen], or None."""
        if self._place_block is None:
            return None
        out = np.empty((self.n_ops, self.n_scen), np.uint16)
        return self._fill(self.place_block, out, threads)

    def columns(self, scen: np.ndarray):
        """Durations (and placements) of the given scenario indices only.

        Returns ``(dur, place)`` with shapes ``[n_ops, len(scen)]``; only the
        blocks that hold those scenarios are generated.
        """
        scen = np.asarray(scen, np.int64)
        dur = np.empty((self.n_ops, scen.size), np.int32)
        place = np.empty((self.n_ops, scen.size), np.uint16) if self.has_place else None
        for b in np.unique(scen // BLOCK):
            sel = np.nonzero(scen // BLOCK == b)[0]
            cols = scen[sel] - b * BLOCK
            dur[:, sel] = self.dur_block(int(b))[:, cols]
            if place is not None:
                place[:, sel] = self.place_block(int(b))[:, cols]
        return dur, place

    def gen_base(self) -> np.ndarray:
        """int32 [n_knobs, n_ops] base durations for on-device generation.

        Scenario s (global index) uses knob ``(s // knob_block) % n_knobs``;
        the generator multiplies the base by a per-(op, scenario) noise
        factor drawn inside the kernel instead of reading ``durations()``.
        """
        if self._gen_base is None:
            raise ValueError(f"{self.name} has no base table")
        return _to_ns(np.array(self._gen_base, np.float64, ndmin=2))

    def manifest(self) -> dict:
        indeg = np.bincount(self.succ_idx, minlength=self.n_ops) if self.n_ops else np.zeros(0)
        m = dict(name=self.name, n_ops=self.n_ops, n_edges=self.n_edges, n_res=self.n_res,
                 n_scen=self.n_scen, seed=self.seed, op_events=self.n_ops * self.n_scen,
                 max_in_degree=int(indeg.max()) if indeg.size else 0,
                 max_out_degree=int(np.diff(self.succ_ptr).max()) if self.n_ops else 0,
                 placement=self.has_place)
        m.update(self.info)
        return m


class _Builder:
    """Collects ops (resource, duration model) and edges, emits CSR."""

    def __init__(self):
        self.res: list[int] = []
        self.tag: list[str] = []
        self.edges: list[tuple[int, int]] = []

    def op(self, res: int, tag: str) -> int:
        self.res.append(res)
        self.tag.append(tag)
        return len(self.res) - 1

    def dep(self, u: int, v: int) -> None:
        self.edges.append((u, v))

    def csr(self):
        n = len(self.res)
        e = np.array(sorted(set(self.edges)), np.int64).reshape(-1, 2)
        if e.size and not (e[:, 0] < e[:, 1]).all():
            raise AssertionError("generator emits ops in topological order")
        counts = np.bincount(e[:, 0], minlength=n) if e.size else np.zeros(n, np.int64)
        ptr = np.zeros(n + 1, np.int64)
        np.cumsum(counts, out=ptr[1:])
        return ptr, e[:, 1].astype(np.int32), np.array(self.res, np.int32)


# ---------------------------------------------------------------------------
# Model templates: forward op lists with a mirrored backward pass.
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class _TOp:
    kind: str
    preds: list
    params: int = 0  # parameters whose gradient this op produces (fp32)
    split: bool = False  # backward is two ops (input grad + weight grad)


def _mirror(fwd: list[_TOp]):
    """Backward pass of a forward template (reverse-mode autodiff shape).

    Every forward op except the loss gets a backward op that needs the
    gradient of its output (from the backward ops of its forward consumers)
    and its own forward activation; ops with ``split`` get an input-gradient
    op and a weight-gradient op.  Returns the backward ops as ``_TOp`` with
    predecessor references ``('f', i)`` (forward op i) or ``('b', j)``, and
    for each forward op the index of the backward op holding its parameter
    gradient.
    """
    n = len(fwd)
    succ = [[] for _ in range(n)]
    for i, t in enumerate(fwd):
        for p in t.preds:
            succ[p].append(i)
    loss = n - 1
    assert fwd[loss].kind == "loss"
    bwd: list[_TOp] = []
    provider = {loss: ("f", loss)}  # who delivers d(loss)/d(input of op i)
    grad_op = {}
    for i in range(n - 2, -1, -1):
        preds = [provider[j] for j in succ[i]] + [("f", i)]
        if fwd[i].split:
            bwd.append(_TOp(fwd[i].kind + "_dgrad", preds))
            dg = len(bwd) - 1
            bwd.append(_TOp(fwd[i].kind + "_wgrad", preds, fwd[i].params))
            grad_op[i] = len(bwd) - 1
            provider[i] = ("b", dg)
        else:
            bwd.append(_TOp(fwd[i].kind + "_bwd", preds, fwd[i].params))
            provider[i] = ("b", len(bwd) - 1)
            if fwd[i].params:
                grad_op[i] = len(bwd) - 1
    return bwd, grad_op


def _instantiate(B: _Builder, fwd, bwd, res: int, prefix: str):
    """Emit one replica's forward + backward ops on resource ``res``."""
    fid = []
    for t in fwd:
        v = B.op(res, prefix + t.kind)
        for p in t.preds:
            B.dep(fid[p], v)
        fid.append(v)
    bid = []
    for t in bwd:
        v = B.op(res, prefix + t.kind)
        for side, j in t.preds:
            B.dep(fid[j] if side == "f" else bid[j], v)
        bid.append(v)
    return fid, bid


def _resnet50_template():
    """ResNet-50: 7x7 stem, bottleneck stages (3, 4, 6, 3), fc 2048x1000.

    53 convolutions + fc; BatchNorm gamma/beta are counted with the
    convolution they follow.  Forward: 175 ops, backward: 228 ops.
    """
    f: list[_TOp] = []

    def add(kind, preds, params=0, split=False):
        f.append(_TOp(kind, list(preds), params, split))
        return len(f) - 1

    x = add("conv", [], 7 * 7 * 3 * 64 + 2 * 64, True)
    x = add("bn", [x])
    x = add("relu", [x])
    x = add("maxpool", [x])
    cin = 64
    for nblk, c in ((3, 64), (4, 128), (6, 256), (3, 512)):
        for i in range(nblk):
            inp = x
            a = add("conv", [inp], cin * c + 2 * c, True)
            a = add("bn", [a])
            a = add("relu", [a])
            a = add("conv", [a], 9 * c * c + 2 * c, True)
            a = add("bn", [a])
            a = add("relu", [a])
            a = add("conv", [a], c * 4 * c + 8 * c, True)
            a = add("bn", [a])
            if i == 0:
                sc = add("conv", [inp], cin * 4 * c + 8 * c, True)
                sc = add("bn", [sc])
            else:
                sc = inp
            s = add("add", [a, sc])
            x = add("relu", [s])
            cin = 4 * c
    x = add("avgpool", [x])
    x = add("fc", [x], 2048 * 1000 + 1000, True)
    add("loss", [x])
    return f


def _inception_v3_template(rng: np.random.Generator, total_params: int = 23_800_000):
    """Inception-v3-like: stem, 11 four-branch modules (3 A, 1 B, 4 C, 1 D, 2 E),
    pool, fc, loss.  Branch lengths per module type are fixed below; parameter
    counts per convolution are random with the model's 23.8 M total."""
    f: list[_TOp] = []

    def add(kind, preds, conv=False):
        f.append(_TOp(kind, list(preds), 1 if conv else 0))
        return len(f) - 1

    x = add("conv", [], True)
    x = add("conv", [x], True)
    x = add("conv", [x], True)
    x = add("pool", [x])
    x = add("conv", [x], True)
    x = add("conv", [x], True)
    x = add("pool", [x])
    # each branch: sequence of 'c' (conv) / 'p' (pool) ops
    mods = {"A": ["c", "cc", "ccc", "pc"], "B": ["cc", "ccc", "p", "c"],
            "C": ["c", "ccc", "ccccc", "pc"], "D": ["cc", "cccc", "p", "c"],
            "E": ["c", "ccc", "cccc", "pc"]}
    for m in "AAABCCCCDEE":
        ends = []
        for br in mods[m]:
            y = x
            for k in br:
                y = add("conv" if k == "c" else "pool", [y], k == "c")
            ends.append(y)
        x = add("concat", ends)
    x = add("avgpool", [x])
    x = add("fc", [x], True)
    add("loss", [x])
    w = _log_uniform(rng, 1.0, 100.0, sum(1 for t in f if t.params))
    w = np.floor(w / w.sum() * total_params).astype(np.int64)
    k = 0
    for t in f:
        if t.params:
            t.params = int(w[k])
            k += 1
    return f


def _bert_large_template():
    """BERT-large encoder: embedding, 24 x (QKV GEMM, softmax, out-proj, LN1,
    FFN1, FFN2, LN2), loss; post-LN residuals.  Forward: 170 ops."""
    h, ff, vocab = 1024, 4096, 30522 + 512 + 2
    f: list[_TOp] = []

    def add(kind, preds, params=0):
        f.append(_TOp(kind, list(preds), params))
        return len(f) - 1

    x = add("embed", [], vocab * h + 2 * h)
    for _ in range(24):
        inp = x
        a = add("qkv", [inp], 3 * h * h + 3 * h)
        a = add("softmax", [a])
        a = add("outproj", [a], h * h + h)
        ln1 = add("ln1", [a, inp], 2 * h)
        a = add("ffn1", [ln1], h * ff + ff)
        a = add("ffn2", [a], ff * h + h)
        x = add("ln2", [a, ln1], 2 * h)
    add("loss", [x])
    return f


# ---------------------------------------------------------------------------
# The five workloads.
# ---------------------------------------------------------------------------

def _noisy(base: np.ndarray, rng: np.random.Generator, sigma: float = 0.01) -> np.ndarray:
    """float64 [n, BLOCK]: base[v] * exp(sigma * Z[v, s]), Z standard normal.

    Z and the factor are single precision (the factor's relative error is
    ~1e-7, far below the 1 % spread it models); the product is double.
    """
    z = rng.standard_normal((base.size, BLOCK), dtype=np.float32)
    z *= np.float32(sigma)
    np.exp(z, out=z)
    return np.multiply(z, base[:, None])


def tiny_dp_mlp(n_scen: int = 1024, seed: int = _SEED_BASE + 1) -> Workload:
    """3 dense layers, 2 data-parallel workers, one shared link.

    Per worker w (resource w): F0 A0 F1 A1 F2 A2 Ab2 B2 Ab1 B1 Ab0 B0 (forward
    GEMM/activation, backward activation/GEMM); B_l -> push P(w,l) on the link
    (resource 2); every P(.,l) -> pull Q(w,l) on the link; Q(w,l) -> update
    U(w,l) on resource w.  42 ops, 46 edges.  Base durations uniform integers
    in [10 us, 1 ms]; every (op, scenario) is perturbed by lognormal(0, 0.01).
    """
    B = _Builder()
    link = 2
    B_op, P = {}, {}
    for w in range(2):
        names = ["F0", "A0", "F1", "A1", "F2", "A2", "Ab2", "B2", "Ab1", "B1", "Ab0", "B0"]
        prev = None
        for nm in names:
            v = B.op(w, f"w{w}.{nm}")
            if prev is not None:
                B.dep(prev, v)
            prev = v
            if nm.startswith("B"):
                B_op[(w, int(nm[1]))] = v
    for w in range(2):
        for l in (2, 1, 0):
            P[(w, l)] = B.op(link, f"push.w{w}.l{l}")
            B.dep(B_op[(w, l)], P[(w, l)])
    Q = {}
    for w in range(2):
        for l in (2, 1, 0):
            Q[(w, l)] = B.op(link, f"pull.w{w}.l{l}")
            for w2 in range(2):
                B.dep(P[(w2, l)], Q[(w, l)])
    for w in range(2):
        for l in (2, 1, 0):
            u = B.op(w, f"upd.w{w}.l{l}")
            B.dep(Q[(w, l)], u)
    ptr, idx, res = B.csr()
    base = _rng(seed, 0).integers(10_000, 1_000_000, size=res.size, endpoint=True).astype(np.float64)
    return Workload("tiny-dp-mlp", res.size, 3, ptr, idx, res, n_scen, seed,
                    _dur_block=lambda b: _noisy(base, _rng(seed, 1, b)),
                    info=dict(workers=2, layers=3), _gen_base=base[None, :])


def resnet50_ps(n_scen: int = 65536, seed: int = _SEED_BASE + 2, workers: int = 8) -> Workload:
    """ResNet-50 data parallel over a parameter server.

    Resources: worker compute 0..W-1, worker link W..2W-1, PS W*2.  Per
    parameter layer l: weight-grad -> push(w,l) on link w -> PS aggregate
    agg(l) (after all W pushes) -> pull(w,l) on link w -> update(w,l).
    Compute bases are log-uniform in [5 us, 5 ms] per template op, shared by
    all workers; push/pull take bytes / 10 GB/s, aggregation 8*bytes / 100 GB/s.
    """
    W = workers
    rng = _rng(seed, 0)
    fwd = _resnet50_template()
    bwd, grad_op = _mirror(fwd)
    nt = len(fwd) + len(bwd)
    tbase = _log_uniform(rng, 5e3, 5e6, nt)
    layers = [i for i in range(len(fwd)) if fwd[i].params]
    ubase = _log_uniform(rng, 5e3, 5e6, len(layers))
    B = _Builder()
    base = []
    grads = {}
    for w in range(W):
        fid, bid = _instantiate(B, fwd, bwd, w, f"w{w}.")
        base.extend(tbase)
        for li, i in enumerate(layers):
            grads[(w, li)] = bid[grad_op[i]]
    nbytes = np.array([4.0 * fwd[i].params for i in layers])
    push = {}
    for w in range(W):
        for li in range(len(layers)):
            push[(w, li)] = B.op(W + w, f"push.w{w}.l{li}")
            B.dep(grads[(w, li)], push[(w, li)])
            base.append(nbytes[li] / 10.0)
    agg = {}
    for li in range(len(layers)):
        agg[li] = B.op(2 * W, f"agg.l{li}")
        for w in range(W):
            B.dep(push[(w, li)], agg[li])
        base.append(8.0 * nbytes[li] / 100.0)
    pull = {}
    for w in range(W):
        for li in range(len(layers)):
            pull[(w, li)] = B.op(W + w, f"pull.w{w}.l{li}")
            B.dep(agg[li], pull[(w, li)])
            base.append(nbytes[li] / 10.0)
    for w in range(W):
        for li in range(len(layers)):
            u = B.op(w, f"upd.w{w}.l{li}")
            B.dep(pull[(w, li)], u)
            base.append(ubase[li])
    ptr, idx, res = B.csr()
    base = np.array(base)
    return Workload("resnet50-ps", res.size, 2 * W + 1, ptr, idx, res, n_scen, seed,
                    _dur_block=lambda b: _noisy(base, _rng(seed, 1, b)),
                    info=dict(workers=W, fwd_ops=len(fwd), bwd_ops=len(bwd),
                              param_layers=len(layers)), _gen_base=base[None, :])


def inception_v3_ring(n_scen: int = 65536, seed: int = _SEED_BASE + 3, devices: int = 4,
                      buckets: int = 4) -> Workload:
    """Inception-v3 data parallel with a ring all-reduce.

    Per device d: compute stream (resource d) and copy stream (resource D+d).
    Input H2D copy on the copy stream; forward + mirrored backward on the
    compute stream.  Gradients fill ``buckets`` equal buckets in backward
    order; bucket b's ring all-reduce is 2(D-1) chunk steps X(b,k,d) on copy
    stream d, each after X(b,k-1,d) and X(b,k-1,d-1); update U(b,d) on the
    compute stream after the last step.  Every base duration is log-uniform
    in [5 us, 5 ms], shared by the replicas.
    """
    D = devices
    rng = _rng(seed, 0)
    fwd = _inception_v3_template(rng)
    bwd, grad_op = _mirror(fwd)
    nt = len(fwd) + len(bwd)
    tbase = _log_uniform(rng, 5e3, 5e6, nt)
    h2d_base = _log_uniform(rng, 5e3, 5e6, 1)[0]
    steps = 2 * (D - 1)
    ring_base = _log_uniform(rng, 5e3, 5e6, (buckets, steps))
    upd_base = _log_uniform(rng, 5e3, 5e6, buckets)
    # buckets in backward order of the weight-gradient ops, equal byte shares
    order = sorted(grad_op.items(), key=lambda kv: kv[1])  # backward emission order
    pbytes = np.array([4.0 * fwd[i].params for i, _ in order])
    cum = np.cumsum(pbytes) - pbytes
    bucket_of = np.minimum((cum / pbytes.sum() * buckets).astype(int), buckets - 1)
    B = _Builder()
    base = []
    members = {}
    for d in range(D):
        h = B.op(D + d, f"d{d}.h2d")
        base.append(h2d_base)
        fid, bid = _instantiate(B, fwd, bwd, d, f"d{d}.")
        B.dep(h, fid[0])
        base.extend(tbase)
        for (i, j), b in zip(order, bucket_of):
            members.setdefault((d, int(b)), []).append(bid[j])
    X = {}
    for b in range(buckets):
        for k in range(steps):
            for d in range(D):
                v = B.op(D + d, f"ring.b{b}.k{k}.d{d}")
                base.append(ring_base[b, k])
                if k == 0:
                    for g in members[(d, b)]:
                        B.dep(g, v)
                else:
                    B.dep(X[(b, k - 1, d)], v)
                    B.dep(X[(b, k - 1, (d - 1) % D)], v)
                X[(b, k, d)] = v
    for b in range(buckets):
        for d in range(D):
            u = B.op(d, f"upd.b{b}.d{d}")
            base.append(upd_base[b])
            B.dep(X[(b, steps - 1, d)], u)
            B.dep(X[(b, steps - 1, (d - 1) % D)], u)
    ptr, idx, res = B.csr()
    base = np.array(base)
    return Workload("inception-v3-ring", res.size, 2 * D, ptr, idx, res, n_scen, seed,
                    _dur_block=lambda b: _noisy(base, _rng(seed, 1, b)),
                    info=dict(devices=D, buckets=buckets, fwd_ops=len(fwd), bwd_ops=len(bwd),
                              bucket_mb=[float(pbytes[bucket_of == b].sum() / 1e6)
                                         for b in range(buckets)]), _gen_base=base[None, :])


#: strategy knobs of the BERT workload: (compute batch factor, link GB/s)
BERT_KNOBS = [(bf, bw) for bf in (0.5, 1.0, 2.0, 4.0) for bw in (10.0, 25.0, 100.0)]


def bert_large_ps(n_scen: int = 262144, seed: int = _SEED_BASE + 4, workers: int = 16) -> Workload:
    """BERT-large data parallel over per-worker up/down links.

    Resources: worker compute 0..W-1, uplink W..2W-1, downlink 2W..3W-1.
    Gradient buckets are the 24 encoder layers plus the embeddings; push(w,b)
    on uplink w after the layer's backward ops, pull(w,b) on downlink w after
    all W pushes of b, update(w,b) on compute w.  Scenario s uses strategy
    knob ``(s // 4096) % 12``: compute bases (log-uniform [5 us, 2 ms], per
    template op, shared by workers) times a batch factor in {0.5, 1, 2, 4};
    push/pull take bytes / bandwidth with bandwidth in {10, 25, 100} GB/s.
    Updates do not scale with the batch.
    """
    W = workers
    rng = _rng(seed, 0)
    fwd = _bert_large_template()
    bwd, grad_op = _mirror(fwd)
    nt = len(fwd) + len(bwd)
    tbase = _log_uniform(rng, 5e3, 2e6, nt)
    nb = 25
    upd_base = _log_uniform(rng, 5e3, 2e6, nb)
    # bucket of each parameterised forward op: its encoder layer, embeddings last
    bucket = {}
    layer = -1
    for i, t in enumerate(fwd):
        if t.kind == "qkv":
            layer += 1
        if t.params:
            bucket[i] = 24 if t.kind == "embed" else layer
    nbytes = np.zeros(nb)
    for i, b in bucket.items():
        nbytes[b] += 4.0 * fwd[i].params
    B = _Builder()
    comp, comm, cls = [], [], []  # per op: compute base, bytes, class (0 batch-scaled, 1 comm, 2 fixed)
    grads = {}
    for w in range(W):
        fid, bid = _instantiate(B, fwd, bwd, w, f"w{w}.")
        comp.extend(tbase)
        comm.extend([0.0] * nt)
        cls.extend([0] * nt)
        for i, b in bucket.items():
            grads.setdefault((w, b), []).append(bid[grad_op[i]])
    push = {}
    for w in range(W):
        for b in range(nb):
            push[(w, b)] = B.op(W + w, f"push.w{w}.b{b}")
            for g in grads[(w, b)]:
                B.dep(g, push[(w, b)])
            comp.append(0.0)
            comm.append(nbytes[b])
            cls.append(1)
    pull = {}
    for w in range(W):
        for b in range(nb):
            pull[(w, b)] = B.op(2 * W + w, f"pull.w{w}.b{b}")
            for w2 in range(W):
                B.dep(push[(w2, b)], pull[(w, b)])
            comp.append(0.0)
            comm.append(nbytes[b])
            cls.append(1)
    for w in range(W):
        for b in range(nb):
            u = B.op(w, f"upd.w{w}.b{b}")
            B.dep(pull[(w, b)], u)
            comp.append(upd_base[b])
            comm.append(0.0)
            cls.append(2)
    ptr, idx, res = B.csr()
    comp, comm, cls = np.array(comp), np.array(comm), np.array(cls)

    def knob_base(bf, bw):
        return np.where(cls == 1, comm / bw, np.where(cls == 0, comp * bf, comp))

    def dur_block(b):
        return _noisy(knob_base(*BERT_KNOBS[(b * BLOCK // 4096) % len(BERT_KNOBS)]), _rng(seed, 1, b))

    assert BLOCK % 4096 == 0 or 4096 % BLOCK == 0
    return Workload("bert-large-ps", res.size, 3 * W, ptr, idx, res, n_scen, seed,
                    _dur_block=dur_block,
                    info=dict(workers=W, buckets=nb, fwd_ops=len(fwd), bwd_ops=len(bwd),
                              knob_block=4096, knobs=BERT_KNOBS,
                              bucket_mb=[float(x / 1e6) for x in nbytes]),
                    _gen_base=np.stack([knob_base(bf, bw) for bf, bw in BERT_KNOBS]), knob_block=4096)


def random_layered(n_scen: int = 16384, seed: int = _SEED_BASE + 5, levels: int = 200,
                   width: int = 100, n_res: int = 64) -> Workload:
    """Random layered DAG with a per-scenario placement.

    ``levels`` x ``width`` ops; each op past level 0 takes 1-4 distinct
    predecessors uniformly from the previous level.  ``op_res`` is uniform over
    ``n_res``; ``place[v, s]`` (uniform, per op and scenario) overrides it.
    Durations are i.i.d. log-uniform in [1 us, 10 ms] per (op, scenario).
    """
    rng = _rng(seed, 0)
    B = _Builder()
    lvl_ops = []
    for L in range(levels):
        ops = [B.op(0, f"L{L}") for _ in range(width)]
        if L:
            for v in ops:
                k = int(rng.integers(1, 5))
                for p in rng.choice(width, size=k, replace=False):
                    B.dep(lvl_ops[-1][int(p)], v)
        lvl_ops.append(ops)
    B.res = list(rng.integers(0, n_res, size=len(B.res)))
    ptr, idx, res = B.csr()
    n = res.size

    def dur_block(b):
        return _log_uniform(_rng(seed, 1, b), 1e3, 1e7, (n, BLOCK))

    def place_block(b):
        return _rng(seed, 2, b).integers(0, n_res, size=(n, BLOCK), dtype=np.uint16)

    return Workload("random-layered", n, n_res, ptr, idx, res, n_scen, seed,
                    _dur_block=dur_block, _place_block=place_block,
                    info=dict(levels=levels, width=width),
                    _gen_base=_log_uniform(_rng(seed, 3), 1e3, 1e7, (1, n)))


CONFIGS = {
    1: tiny_dp_mlp,
    2: resnet50_ps,
    3: inception_v3_ring,
    4: bert_large_ps,
    5: random_layered,
}


def link_resources(w: Workload) -> np.ndarray:
    """Resources of ``w`` that carry transfers (candidates for bandwidth
    sharing): the tiny model's shared link, the workers' links of the
    parameter-server graphs, the copy streams of the ring graph; none for
    the random layered graph."""
    name, info = w.name, w.info
    if name.startswith("tiny-dp-mlp"):
        return np.array([2])
    if name.startswith("resnet50-ps"):
        return np.arange(info["workers"], 2 * info["workers"])
    if name.startswith("inception-v3-ring"):
        return np.arange(info["devices"], 2 * info["devices"])
    if name.startswith("bert-large-ps"):
        return np.arange(info["workers"], 3 * info["workers"])
    return np.zeros(0, np.int64)


def make_config(k: int, n_scen: Optional[int] = None) -> Workload:
    """Workload k (1..5) at its full scenario count, or at ``n_scen``."""
    fn = CONFIGS[k]
    return fn() if n_scen is None else fn(n_scen=n_scen)


# ---------------------------------------------------------------------------
# Small random graphs for tests.
# ---------------------------------------------------------------------------

def random_dag(n: int, n_res: int, edge_p: float, rng: np.random.Generator,
               shuffle_ids: bool = True, with_prio: bool = False, dup_edges: bool = False):
    """Random DAG (n ops, Bernoulli(edge_p) forward edges) with random op ids.

    Returns (succ_ptr int64, succ_idx int32, op_res int32, prio int32|None).
    Successor lists are unsorted; with ``dup_edges`` some edges repeat.
    """
    a = np.triu(rng.random((n, n)) < edge_p, 1)
    perm = rng.permutation(n) if shuffle_ids else np.arange(n)
    us, vs = np.nonzero(a)
    us, vs = perm[us], perm[vs]
    if dup_edges and us.size:
        k = rng.integers(0, us.size, size=max(1, us.size // 4))
        us, vs = np.concatenate([us, us[k]]), np.concatenate([vs, vs[k]])
    order = rng.permutation(us.size)
    us, vs = us[order], vs[order]
    srt = np.argsort(us, kind="stable")
    us, vs = us[srt], vs[srt]
    counts = np.bincount(us, minlength=n)
    ptr = np.zeros(n + 1, np.int64)
    np.cumsum(counts, out=ptr[1:])
    res = rng.integers(0, n_res, size=n).astype(np.int32)
    prio = rng.integers(-3, 4, size=n).astype(np.int32) if with_prio else None
    return ptr, vs.astype(np.int32), res, prio


def random_durations(n: int, n_scen: int, lo: int, hi: int, rng: np.random.Generator) -> np.ndarray:
    """int32 [n, n_scen] uniform integers in [lo, hi]."""
    return rng.integers(lo, hi, size=(n, n_scen), endpoint=True).astype(np.int32)
