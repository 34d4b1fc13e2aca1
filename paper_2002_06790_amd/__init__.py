"""Batched dataflow replay of ML training iterations on AMD MI355X.

Python binding of ``libmlsim.so`` (C ABI declared in ``include/mlsim.h``).
This module only marshals arguments: every step of the replay runs in the
library's HIP kernels.  PyTorch supplies device memory and the stream.

The replay follows the paper's simulation module (Huang et al., "Simulating
Performance of ML Systems with Offline Profiling", Sec. 2, "Dataflow based
simulation"): each device or link runs its ready ops one at a time, first in
first out by ready time, and the iteration time is the finish time of the
last device.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmlsim.so")

SIM_OK, SIM_E_INVAL, SIM_E_RANGE, SIM_E_CYCLE, SIM_E_NOMEM, SIM_E_HIP, SIM_E_LIMIT = 0, -1, -2, -3, -4, -5, -6
SIM_ST_BAD_DUR, SIM_ST_BAD_RES, SIM_ST_OVERFLOW, SIM_ST_SHARE_LIMIT, SIM_ST_INTERNAL = 1, 2, 4, 8, 16
#: bandwidth sharing (include/mlsim.h): most active ops per shared resource, service units per ns
SIM_SHARE_MAX, SIM_SHARE_UNIT = 64, 2952069120
SIM_ALGO_AUTO, SIM_ALGO_EVENT, SIM_ALGO_SWEEP = 0, 1, 2
ALGOS = {"auto": SIM_ALGO_AUTO, "event": SIM_ALGO_EVENT, "sweep": SIM_ALGO_SWEEP}
#: kernel-variant pins of the testing entry point (include/mlsim_testing.h)
TEST_VARIANTS = {"auto": 0, "ev_lds_groups": 1, "ev_blocks_cap": 3, "ev_reg": 4, "cp_global": 5,
                 "rf_global": 6, "share_key_id": 7}

EXPORTS = ("sim_graph_create", "sim_graph_destroy", "sim_run_batch", "sim_critical_path",
           "sim_strerror", "sim_graph_info", "sim_testing_replan", "sim_static_create",
           "sim_static_destroy", "sim_static_run", "sim_attribute", "sim_generate", "sim_run_generated",
           "sim_critical_path_generated", "sim_run_batch_gap", "sim_static_run_generated",
           "sim_run_batch_dev", "sim_run_batch_share", "sim_run_batch_noalloc", "sim_testing_sweep_table",
           "sim_testing_join_slots")

#: generator limits (include/mlsim.h): largest base duration, noise bound
SIM_GEN_BASE_MAX, SIM_GEN_NOISE_MAX = 1 << 24, 1 << 20
#: relative standard deviation of the generated noise per unit of ``noise``
GEN_SIGMA_UNIT = 2.0 * (2.0 * (65536.0**2 - 1.0) / 3.0) ** 0.5 / 2.0**40

_lib = None


class SimError(RuntimeError):
    def __init__(self, code: int, what: str = ""):
        msg = _load().sim_strerror(code).decode() if _lib is not None else str(code)
        super().__init__(f"{what}: {msg} ({code})" if what else f"{msg} ({code})")
        self.code = code


def build() -> str:
    """Compile libmlsim.so for gfx950 (always rebuilds)."""
    from . import buildlib as _b
    global _lib
    path = _b.build()
    _lib = None
    return path


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built: call paper_2002_06790_amd.build()")
    L = ctypes.CDLL(LIB_PATH)
    P, I32, I64, U32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32
    L.sim_graph_create.argtypes = [I32, I32, P, P, P, P, ctypes.POINTER(P)]
    L.sim_graph_create.restype = ctypes.c_int
    L.sim_graph_destroy.argtypes = [P]
    L.sim_graph_destroy.restype = None
    L.sim_run_batch.argtypes = [P, I64, P, I64, P, I64, P, P, I64, P, U32, P]
    L.sim_run_batch.restype = ctypes.c_int
    L.sim_critical_path.argtypes = [P, I64, P, I64, P, I64, P, I32, P, P]
    L.sim_critical_path.restype = ctypes.c_int
    L.sim_strerror.argtypes = [ctypes.c_int]
    L.sim_strerror.restype = ctypes.c_char_p
    L.sim_graph_info.argtypes = [P, P, P, P, P, P]
    L.sim_graph_info.restype = ctypes.c_int
    L.sim_testing_replan.argtypes = [P, I32, I32]
    L.sim_testing_replan.restype = ctypes.c_int
    L.sim_static_create.argtypes = [P, P, ctypes.POINTER(P)]
    L.sim_static_create.restype = ctypes.c_int
    L.sim_static_destroy.argtypes = [P]
    L.sim_static_destroy.restype = None
    L.sim_static_run.argtypes = [P, I64, P, I64, P, P, I64, P, P]
    L.sim_static_run.restype = ctypes.c_int
    L.sim_attribute.argtypes = [P, I64, P, I64, P, I64, P, P, P, P, I64, P, P, I64, P, I64, P, I32, P, P]
    L.sim_attribute.restype = ctypes.c_int
    U64 = ctypes.c_uint64
    L.sim_generate.argtypes = [I32, I64, P, I32, I64, U32, U64, I64, P, I64, P]
    L.sim_generate.restype = ctypes.c_int
    L.sim_run_generated.argtypes = [P, I64, P, I32, I64, U32, U64, I64, P, P, I64, P, U32, P]
    L.sim_run_generated.restype = ctypes.c_int
    L.sim_critical_path_generated.argtypes = [P, I64, P, I32, I64, U32, U64, I64, P, I64, P, I32, P, P]
    L.sim_critical_path_generated.restype = ctypes.c_int
    L.sim_run_batch_gap.argtypes = [P, I64, P, I64, P, I64, P, P, P, I64, P, U32, P]
    L.sim_run_batch_gap.restype = ctypes.c_int
    L.sim_run_batch_dev.argtypes = [P, I64, P, I64, P, I64, P, P, P, P, I64, P, U32, P]
    L.sim_run_batch_dev.restype = ctypes.c_int
    L.sim_run_batch_noalloc.argtypes = [P, I64, P, I64, P, I64, P, P, I64, P, U32, P]
    L.sim_run_batch_noalloc.restype = ctypes.c_int
    L.sim_run_batch_share.argtypes = [P, I64, P, I64, P, P, P, I64, P, P]
    L.sim_run_batch_share.restype = ctypes.c_int
    L.sim_static_run_generated.argtypes = [P, I64, P, I32, I64, U32, U64, I64, P, P, I64, P, P]
    L.sim_static_run_generated.restype = ctypes.c_int
    L.sim_testing_sweep_table.argtypes = [I32, I32, P, P, P, P, P, P, P, P, I64, P, I64, P]
    L.sim_testing_sweep_table.restype = ctypes.c_int
    L.sim_testing_join_slots.argtypes = [I32, I32, P, P, P, P, P, P]
    L.sim_testing_join_slots.restype = ctypes.c_int
    _lib = L
    return L


def lib():
    """The loaded ctypes library (raises if it is not built)."""
    return _load()


def sweep_table(succ_ptr, succ_idx, op_res, n_res: int, prio=None, order=None):
    """The max-plus sweep table the library builds for a graph, on the host
    only (sim_testing_sweep_table): the critical-path table, or with
    ``order`` (a permutation of the op ids) the static-order replay's.
    Returns ``(rec int32 [n_rec, 8], plist int32, slots)``; the fields of a
    record are {row, slot, npred, pbeg, p0, p1, p2, p3} (row -1: a barrier
    record)."""
    L = _load()
    ptr = _host(succ_ptr, np.int64)
    idx = _host(succ_idx, np.int32)
    res = _host(op_res, np.int32)
    pr = _host(prio, np.int32)
    od = _host(order, np.int32)
    n = int(ptr.size - 1)
    if res.size != n or (pr is not None and pr.size != n) or (od is not None and od.size != n):
        raise ValueError("op_res, prio and order need one entry per op")
    n_rec, slots, plen = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int64()
    rec = np.zeros((0, 8), np.int32)
    plist = np.zeros(0, np.int32)
    for _ in range(2):  # sizes first, then the table
        rc = L.sim_testing_sweep_table(n, int(n_res), _hptr(ptr), _hptr(idx), _hptr(res), _hptr(pr), _hptr(od),
                                       ctypes.byref(n_rec), ctypes.byref(slots), _hptr(rec) if rec.size else None,
                                       rec.shape[0], _hptr(plist) if plist.size else None, plist.size,
                                       ctypes.byref(plen))
        if rc == SIM_OK:
            return rec[:n_rec.value].copy(), plist[:plen.value].copy(), slots.value
        if rc != SIM_E_LIMIT or (rec.shape[0] >= n_rec.value and plist.size >= plen.value):
            raise SimError(rc, "sim_testing_sweep_table")
        rec = np.zeros((n_rec.value, 8), np.int32)
        plist = np.zeros(max(plen.value, 1), np.int32)
    raise SimError(SIM_E_LIMIT, "sim_testing_sweep_table")


def join_slots(succ_ptr, succ_idx, op_res, n_res: int, prio=None):
    """The event replay's join state slots for a graph, on the host only
    (sim_testing_join_slots).  Returns ``(slot_of int32 [n_ops], n_slots)``:
    the slot of the join each op waits on (-1: none)."""
    L = _load()
    ptr = _host(succ_ptr, np.int64)
    idx = _host(succ_idx, np.int32)
    res = _host(op_res, np.int32)
    pr = _host(prio, np.int32)
    n = int(ptr.size - 1)
    if res.size != n or (pr is not None and pr.size != n):
        raise ValueError("op_res and prio need one entry per op")
    slot_of = np.full(max(n, 1), -2, np.int32)
    n_slots = ctypes.c_int32()
    rc = L.sim_testing_join_slots(n, int(n_res), _hptr(ptr), _hptr(idx), _hptr(res), _hptr(pr),
                                  _hptr(slot_of), ctypes.byref(n_slots))
    if rc != SIM_OK:
        raise SimError(rc, "sim_testing_join_slots")
    return slot_of[:n].copy(), n_slots.value


def _host(a, dt):
    return None if a is None else np.ascontiguousarray(np.asarray(a), dtype=dt)


def _hptr(a):
    return None if a is None else a.ctypes.data


def _dev_matrix(t, dtype, n_ops, what):
    """(pointer, ld) of a [n_ops, S] device tensor with unit column stride."""
    import torch
    if t is None:
        return None, 0
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{what} must be a torch tensor on the GPU")
    if t.dtype != dtype or t.dim() != 2 or t.shape[0] != n_ops:
        raise ValueError(f"{what} must be {dtype} of shape (n_ops={n_ops}, n_scen)")
    if t.shape[1] > 1 and t.stride(1) != 1:
        raise ValueError(f"{what} must have unit stride along scenarios")
    if n_ops > 1 and t.shape[1] > 0 and t.stride(0) < t.shape[1]:
        raise ValueError(f"{what}: rows overlap (row stride {t.stride(0)} < {t.shape[1]} scenarios)")
    return t.data_ptr(), max(t.stride(0), t.shape[1])


def _dev_vector(t, n, what, device=None):
    """Pointer of a caller-supplied int32 [>= n] device vector with unit stride."""
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{what} must be a torch tensor on the GPU")
    if t.dtype != torch.int32 or t.dim() != 1 or t.numel() < n:
        raise ValueError(f"{what} must be int32 of shape ({n},) or longer")
    if n > 1 and t.stride(0) != 1:
        raise ValueError(f"{what} must be contiguous")
    if device is not None and t.device != device:
        raise ValueError(f"{what} is on {t.device}, the inputs on {device}")
    return t.data_ptr()


def _dev_out_matrix(t, n_ops, n, what, device):
    """(pointer, ld) of a caller-supplied int32 [n_ops, >= n] output matrix."""
    import torch
    p, ld = _dev_matrix(t, torch.int32, n_ops, what)
    if t is not None and (t.shape[1] < n or t.device != device):
        raise ValueError(f"{what} must hold {n} scenarios on {device}")
    return p, ld


def noise_for_sigma(sigma: float) -> int:
    """The generator's ``noise`` argument for a relative standard deviation."""
    noise = int(round(sigma / GEN_SIGMA_UNIT))
    if not 0 <= noise < SIM_GEN_NOISE_MAX:
        raise ValueError(f"sigma {sigma} outside the generator's range")
    return noise


class Gen:
    """Parameters of on-device scenario generation (include/mlsim.h).

    ``base``: int32 [n_knobs, n_ops] device tensor of base durations per
    strategy knob; global scenario S uses knob ``(S // knob_block) % n_knobs``
    and multiplies each base by counter-based noise of relative standard
    deviation ``noise * GEN_SIGMA_UNIT`` keyed by ``seed``; ``scen0`` is the
    global index of the call's first scenario.
    """

    def __init__(self, base, knob_block: int = 1, noise: int = 0, seed: int = 0, scen0: int = 0):
        import torch
        if not isinstance(base, torch.Tensor) or not base.is_cuda or base.dtype != torch.int32:
            raise TypeError("base must be an int32 torch tensor on the GPU")
        if base.dim() == 1:
            base = base[None, :]
        self.base = base.contiguous()
        self.n_knobs, self.n_ops = int(self.base.shape[0]), int(self.base.shape[1])
        self.knob_block, self.noise, self.seed, self.scen0 = int(knob_block), int(noise), int(seed), int(scen0)

    def args(self):
        return (self.base.data_ptr(), self.n_knobs, self.knob_block, self.noise,
                self.seed & (2**64 - 1), self.scen0)


def generate(gen: Gen, n_scen: int, out=None, stream=None):
    """The generated durations, int32 [n_ops, n_scen] on the GPU (sim_generate)."""
    import torch
    if out is None:
        out = torch.empty((gen.n_ops, n_scen), dtype=torch.int32, device=gen.base.device)
    optr, ld = _dev_out_matrix(out, gen.n_ops, n_scen, "out", gen.base.device)
    rc = _load().sim_generate(gen.n_ops, n_scen, *gen.args(), optr, ld, _stream_ptr(stream))
    if rc:
        raise SimError(rc, "sim_generate")
    return out


def _stream_ptr(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


class Graph:
    """A compiled dataflow graph on the current HIP device (sim_graph_create)."""

    def __init__(self, succ_ptr, succ_idx, op_res, n_res: int, prio=None):
        L = _load()
        self.succ_ptr = _host(succ_ptr, np.int64)
        self.succ_idx = _host(succ_idx, np.int32)
        self.op_res = _host(op_res, np.int32)
        self.prio = _host(prio, np.int32)
        self.n_ops = int(self.op_res.size)
        self.n_res = int(n_res)
        h = ctypes.c_void_p()
        rc = L.sim_graph_create(self.n_ops, self.n_res, _hptr(self.succ_ptr), _hptr(self.succ_idx),
                                _hptr(self.op_res), _hptr(self.prio), ctypes.byref(h))
        if rc:
            raise SimError(rc, "sim_graph_create")
        self._h = h

    @classmethod
    def from_workload(cls, w) -> "Graph":
        return cls(w.succ_ptr, w.succ_idx, w.op_res, w.n_res, prio=w.prio)

    def close(self):
        if getattr(self, "_h", None):
            _load().sim_graph_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def info(self) -> dict:
        vals = [ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int64(), ctypes.c_int32(), ctypes.c_int32()]
        rc = _load().sim_graph_info(self._h, *[ctypes.byref(v) for v in vals])
        if rc:
            raise SimError(rc, "sim_graph_info")
        return dict(zip(("n_ops", "n_res", "n_edges", "n_joins", "n_levels"), [v.value for v in vals]))

    def pin_variant(self, what: str, value: int = 0) -> None:
        """Testing: pin this graph's kernels to one variant (``what`` in
        ``TEST_VARIANTS``; "auto" forgets every pin) and plan its scratch
        again (sim_testing_replan; synchronises the device)."""
        rc = _load().sim_testing_replan(self._h, TEST_VARIANTS[what], int(value))
        if rc:
            raise SimError(rc, "sim_testing_replan")

    def run(self, dur, place=None, want_finish: bool = False, algo: str = "auto",
            makespan=None, finish=None, status=None, stream=None, gap=None, delay=None):
        """Replay every scenario column of ``dur`` (int32 [n_ops, S] on the GPU).

        ``gap`` (host int32 [n_res], or None): each resource's idle time
        between consecutive ops (sim_run_batch_gap; event algorithm only).
        ``delay`` (host int32 [n_res], or None): the time from an op's finish
        on each resource until its outputs reach its successors
        (sim_run_batch_dev, with ``gap`` if given; event algorithm only).

        Returns ``(makespan [S], finish [n_ops, S] or None, status [S])`` as
        device tensors (allocated unless passed in).  Asynchronous on the
        current stream.
        """
        import torch
        dptr, ld = _dev_matrix(dur, torch.int32, self.n_ops, "dur")
        S = dur.shape[1]
        pptr, ldp = _dev_matrix(place, torch.uint16, self.n_ops, "place")
        dev = dur.device
        if place is not None and (place.shape[1] < S or place.device != dev):
            raise ValueError(f"place must hold {S} scenarios on {dev}")
        if makespan is None:
            makespan = torch.empty(S, dtype=torch.int32, device=dev)
        if status is None:
            status = torch.empty(S, dtype=torch.int32, device=dev)
        if want_finish and finish is None:
            finish = torch.empty((self.n_ops, S), dtype=torch.int32, device=dev)
        fptr, ldf = _dev_out_matrix(finish, self.n_ops, S, "finish", dev)
        _dev_vector(makespan, S, "makespan", dev)
        _dev_vector(status, S, "status", dev)
        def _res_vec(x, name):
            x = _host(x, np.int32)
            if x.shape != (self.n_res,):
                raise ValueError(f"{name} must have shape (n_res={self.n_res},)")
            return x

        if delay is not None:
            g = None if gap is None else _res_vec(gap, "gap")
            d = _res_vec(delay, "delay")
            rc = _load().sim_run_batch_dev(self._h, S, dptr, ld, pptr, ldp, _hptr(g), _hptr(d), makespan.data_ptr(),
                                           fptr, ldf, status.data_ptr(), ALGOS[algo], _stream_ptr(stream))
            if rc:
                raise SimError(rc, "sim_run_batch_dev")
        elif gap is None:
            rc = _load().sim_run_batch(self._h, S, dptr, ld, pptr, ldp, makespan.data_ptr(), fptr, ldf,
                                       status.data_ptr(), ALGOS[algo], _stream_ptr(stream))
            if rc:
                raise SimError(rc, "sim_run_batch")
        else:
            g = _res_vec(gap, "gap")
            rc = _load().sim_run_batch_gap(self._h, S, dptr, ld, pptr, ldp, _hptr(g), makespan.data_ptr(), fptr,
                                           ldf, status.data_ptr(), ALGOS[algo], _stream_ptr(stream))
            if rc:
                raise SimError(rc, "sim_run_batch_gap")
        return makespan, finish, status

    def run_share(self, dur, share, want_finish: bool = False, makespan=None, finish=None, status=None,
                  stream=None):
        """Replay every scenario column of ``dur`` with bandwidth sharing on
        the resources where ``share`` (host [n_res], nonzero: shared) is set
        (sim_run_batch_share).  Returns ``(makespan, finish or None, status)``.
        """
        import torch
        dptr, ld = _dev_matrix(dur, torch.int32, self.n_ops, "dur")
        S = dur.shape[1]
        dev = dur.device
        sh = np.ascontiguousarray(np.asarray(share) != 0, dtype=np.uint8)
        if sh.shape != (self.n_res,):
            raise ValueError(f"share must have shape (n_res={self.n_res},)")
        if makespan is None:
            makespan = torch.empty(S, dtype=torch.int32, device=dev)
        if status is None:
            status = torch.empty(S, dtype=torch.int32, device=dev)
        if want_finish and finish is None:
            finish = torch.empty((self.n_ops, S), dtype=torch.int32, device=dev)
        fptr, ldf = _dev_out_matrix(finish, self.n_ops, S, "finish", dev)
        _dev_vector(makespan, S, "makespan", dev)
        _dev_vector(status, S, "status", dev)
        rc = _load().sim_run_batch_share(self._h, S, dptr, ld, _hptr(sh), makespan.data_ptr(), fptr, ldf,
                                         status.data_ptr(), _stream_ptr(stream))
        if rc:
            raise SimError(rc, "sim_run_batch_share")
        return makespan, finish, status

    def run_generated(self, gen: Gen, n_scen: int, want_finish: bool = False, algo: str = "auto",
                      makespan=None, finish=None, status=None, stream=None):
        """Replay ``n_scen`` scenarios whose durations the kernel generates
        from ``gen`` (sim_run_generated); returns ``(makespan, finish or
        None, status)`` as device tensors."""
        import torch
        if gen.n_ops != self.n_ops:
            raise ValueError("base table does not match the graph's op count")
        dev = gen.base.device
        if makespan is None:
            makespan = torch.empty(n_scen, dtype=torch.int32, device=dev)
        if status is None:
            status = torch.empty(n_scen, dtype=torch.int32, device=dev)
        if want_finish and finish is None:
            finish = torch.empty((self.n_ops, n_scen), dtype=torch.int32, device=dev)
        fptr, ldf = _dev_out_matrix(finish, self.n_ops, n_scen, "finish", dev)
        _dev_vector(makespan, n_scen, "makespan", dev)
        _dev_vector(status, n_scen, "status", dev)
        rc = _load().sim_run_generated(self._h, n_scen, *gen.args(), makespan.data_ptr(), fptr, ldf,
                                       status.data_ptr(), ALGOS[algo], _stream_ptr(stream))
        if rc:
            raise SimError(rc, "sim_run_generated")
        return makespan, finish, status

    def critical_path_generated(self, gen: Gen, n_scen: int, path_scen: int = -1, cp_len=None,
                                stream=None):
        """Longest path per generated scenario (sim_critical_path_generated)."""
        import torch
        if gen.n_ops != self.n_ops:
            raise ValueError("base table does not match the graph's op count")
        if cp_len is None:
            cp_len = torch.empty(n_scen, dtype=torch.int32, device=gen.base.device)
        _dev_vector(cp_len, n_scen, "cp_len", gen.base.device)
        cap = max(self.n_ops, 1)
        path = np.empty(cap, np.int32)
        plen = np.zeros(1, np.int32)
        want = path_scen >= 0
        rc = _load().sim_critical_path_generated(self._h, n_scen, *gen.args(), cp_len.data_ptr(), path_scen,
                                                 path.ctypes.data if want else None, cap if want else 0,
                                                 plen.ctypes.data if want else None, _stream_ptr(stream))
        if rc:
            raise SimError(rc, "sim_critical_path_generated")
        return cp_len, (path[: int(plen[0])].copy() if want else None)

    def static_order(self, order) -> "StaticReplay":
        """A static-order replay of this graph: every resource runs its ops
        in the order they appear in ``order`` (a permutation of the op ids)."""
        return StaticReplay(self, order)

    def attribute(self, dur, place=None, path_scen: int = -1, stream=None) -> dict:
        """Replay every scenario column of ``dur`` and attribute its
        iteration time (sim_attribute).  Returns a dict of device tensors
        ``makespan``, ``status``, ``finish``, ``prev`` (op that ran before each
        op on its resource), ``busy`` and ``chain`` ([n_res, S]: busy time and
        binding-chain time per resource), ``chain_ops`` ([S]), and ``path``
        (host array, the binding chain of ``path_scen``, or None)."""
        import torch
        dptr, ld = _dev_matrix(dur, torch.int32, self.n_ops, "dur")
        S = dur.shape[1]
        pptr, ldp = _dev_matrix(place, torch.uint16, self.n_ops, "place")
        dev = dur.device
        if place is not None and (place.shape[1] < S or place.device != dev):
            raise ValueError(f"place must hold {S} scenarios on {dev}")
        out = {k: torch.empty(S, dtype=torch.int32, device=dev) for k in ("makespan", "status", "chain_ops")}
        out["finish"] = torch.empty((self.n_ops, S), dtype=torch.int32, device=dev)
        out["prev"] = torch.empty((self.n_ops, S), dtype=torch.int32, device=dev)
        out["busy"] = torch.empty((self.n_res, S), dtype=torch.int32, device=dev)
        out["chain"] = torch.empty((self.n_res, S), dtype=torch.int32, device=dev)
        cap = max(self.n_ops, 1)
        path = np.empty(cap, np.int32)
        plen = np.zeros(1, np.int32)
        want = path_scen >= 0
        rc = _load().sim_attribute(self._h, S, dptr, ld, pptr, ldp, out["makespan"].data_ptr(),
                                   out["status"].data_ptr(), out["finish"].data_ptr(), out["prev"].data_ptr(),
                                   max(S, 1), out["busy"].data_ptr(), out["chain"].data_ptr(), max(S, 1),
                                   out["chain_ops"].data_ptr(), path_scen, path.ctypes.data if want else None,
                                   cap if want else 0, plen.ctypes.data if want else None, _stream_ptr(stream))
        if rc:
            raise SimError(rc, "sim_attribute")
        out["path"] = path[: int(plen[0])].copy() if want else None
        return out

    def critical_path(self, dur, path_scen: int = -1, cp_len=None, stream=None):
        """Longest path per scenario; with ``path_scen`` >= 0 also its op list."""
        import torch
        dptr, ld = _dev_matrix(dur, torch.int32, self.n_ops, "dur")
        S = dur.shape[1]
        if cp_len is None:
            cp_len = torch.empty(S, dtype=torch.int32, device=dur.device)
        _dev_vector(cp_len, S, "cp_len", dur.device)
        cap = max(self.n_ops, 1)
        path = np.empty(cap, np.int32)
        plen = np.zeros(1, np.int32)
        want = path_scen >= 0
        rc = _load().sim_critical_path(self._h, S, dptr, ld, cp_len.data_ptr(), path_scen,
                                       path.ctypes.data if want else None, cap if want else 0,
                                       plen.ctypes.data if want else None, _stream_ptr(stream))
        if rc:
            raise SimError(rc, "sim_critical_path")
        return cp_len, (path[: int(plen[0])].copy() if want else None)


class StaticReplay:
    """Static-order replay compiled against a graph (sim_static_create)."""

    def __init__(self, graph: Graph, order):
        L = _load()
        self.n_ops = graph.n_ops
        self.order = _host(order, np.int32)
        h = ctypes.c_void_p()
        rc = L.sim_static_create(graph._h, _hptr(self.order), ctypes.byref(h))
        if rc:
            raise SimError(rc, "sim_static_create")
        self._h = h

    def close(self):
        if getattr(self, "_h", None):
            _load().sim_static_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def run(self, dur, want_finish: bool = False, makespan=None, finish=None, status=None, stream=None):
        """Replay every scenario column of ``dur`` (int32 [n_ops, S] on the
        GPU); returns ``(makespan [S], finish [n_ops, S] or None, status [S])``
        as device tensors.  Asynchronous on the current stream."""
        import torch
        dptr, ld = _dev_matrix(dur, torch.int32, self.n_ops, "dur")
        S = dur.shape[1]
        dev = dur.device
        if makespan is None:
            makespan = torch.empty(S, dtype=torch.int32, device=dev)
        if status is None:
            status = torch.empty(S, dtype=torch.int32, device=dev)
        if want_finish and finish is None:
            finish = torch.empty((self.n_ops, S), dtype=torch.int32, device=dev)
        fptr, ldf = _dev_out_matrix(finish, self.n_ops, S, "finish", dev)
        _dev_vector(makespan, S, "makespan", dev)
        _dev_vector(status, S, "status", dev)
        rc = _load().sim_static_run(self._h, S, dptr, ld, makespan.data_ptr(), fptr, ldf,
                                    status.data_ptr(), _stream_ptr(stream))
        if rc:
            raise SimError(rc, "sim_static_run")
        return makespan, finish, status

    def run_generated(self, gen: Gen, n_scen: int, want_finish: bool = False, makespan=None, finish=None,
                      status=None, stream=None):
        """The static-order replay of ``n_scen`` scenarios whose durations the
        kernel generates from ``gen`` (sim_static_run_generated)."""
        import torch
        if gen.n_ops != self.n_ops:
            raise ValueError("base table does not match the graph's op count")
        dev = gen.base.device
        if makespan is None:
            makespan = torch.empty(n_scen, dtype=torch.int32, device=dev)
        if status is None:
            status = torch.empty(n_scen, dtype=torch.int32, device=dev)
        if want_finish and finish is None:
            finish = torch.empty((self.n_ops, n_scen), dtype=torch.int32, device=dev)
        fptr, ldf = _dev_out_matrix(finish, self.n_ops, n_scen, "finish", dev)
        _dev_vector(makespan, n_scen, "makespan", dev)
        _dev_vector(status, n_scen, "status", dev)
        rc = _load().sim_static_run_generated(self._h, n_scen, *gen.args(), makespan.data_ptr(), fptr, ldf,
                                              status.data_ptr(), _stream_ptr(stream))
        if rc:
            raise SimError(rc, "sim_static_run_generated")
        return makespan, finish, status
