"""CPU oracle for the batched dataflow replay -- TEST INFRASTRUCTURE ONLY.

Python side of ``oracle.c`` (ctypes, host numpy arrays).  Only ``tests/``,
``__graft_entry__.smoke()`` and the benchmark's CPU-baseline leg use it; the
library never imports it.  See ``oracle.h`` for the semantics.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboracle.so")

OK, E_INVAL, E_RANGE, E_CYCLE, E_NOMEM = 0, -1, -2, -3, -4
ST_BAD_DUR, ST_BAD_RES, ST_OVERFLOW, ST_SHARE_LIMIT = 1, 2, 4, 8
#: bandwidth sharing: most ops at once on a shared device; service units per ns
SHARE_MAX, SHARE_UNIT = 64, 2952069120


#: sanitizer flags of a checking build (address and undefined-behaviour
#: sanitizers; any undefined behaviour aborts instead of printing and going on)
SANITIZE_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                  "-fno-sanitize-recover=all"]


def build(sanitize: bool = False, out: Optional[str] = None) -> str:
    """Compile ``oracle.c`` with gcc into ``liboracle.so`` (always rebuilds).

    ``sanitize=True`` builds a checking copy with AddressSanitizer and
    UndefinedBehaviorSanitizer instead (``out``, default
    ``liboracle_san.so``); a process that loads it must have the sanitizer
    runtimes preloaded (``sanitizer_env()``).
    """
    out = out or (os.path.join(HERE, "liboracle_san.so") if sanitize else LIB)
    opt = SANITIZE_FLAGS if sanitize else ["-O2"]
    tmp = out + ".tmp"
    subprocess.check_call(["gcc", *opt, "-std=c11", "-Wall", "-Wextra", "-fPIC", "-shared",
                           "-pthread", os.path.join(HERE, "oracle.c"), "-o", tmp])
    os.replace(tmp, out)
    return out


def sanitizer_env(path: str) -> dict:
    """Environment for a child process whose oracle calls go to the
    sanitized build at ``path`` (runtimes preloaded, errors fatal)."""
    rt = [subprocess.check_output(["gcc", f"-print-file-name={name}"], text=True).strip()
          for name in ("libasan.so", "libubsan.so")]
    env = dict(os.environ)
    env["LD_PRELOAD"] = ":".join(rt + ([env["LD_PRELOAD"]] if env.get("LD_PRELOAD") else []))
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["ORACLE_LIB"] = path
    return env


_lib = None


def lib(path: Optional[str] = None):
    """The loaded oracle library (``path`` loads another build of oracle.c)."""
    global _lib
    if path is None and _lib is None and os.environ.get("ORACLE_LIB"):
        path = os.environ["ORACLE_LIB"]  # a checking build (sanitizer_env)
        _lib = lib(path)
        return _lib
    if path is not None or _lib is None:
        if path is None and not os.path.exists(LIB):
            build()
        L = ctypes.CDLL(path or LIB)
        P = ctypes.c_void_p
        L.oracle_run_batch.argtypes = [ctypes.c_int32, ctypes.c_int32, P, P, P, P, ctypes.c_int64,
                                       P, ctypes.c_int64, P, ctypes.c_int64, P, P, ctypes.c_int64,
                                       P, ctypes.c_int32]
        L.oracle_run_batch.restype = ctypes.c_int
        L.oracle_run_batch_gap.argtypes = [ctypes.c_int32, ctypes.c_int32, P, P, P, P, P, ctypes.c_int64,
                                           P, ctypes.c_int64, P, ctypes.c_int64, P, P, ctypes.c_int64,
                                           P, ctypes.c_int32]
        L.oracle_run_batch_gap.restype = ctypes.c_int
        L.oracle_run_batch_dev.argtypes = [ctypes.c_int32, ctypes.c_int32, P, P, P, P, P, P, ctypes.c_int64,
                                           P, ctypes.c_int64, P, ctypes.c_int64, P, P, ctypes.c_int64,
                                           P, ctypes.c_int32]
        L.oracle_run_batch_dev.restype = ctypes.c_int
        L.oracle_run_batch_share.argtypes = [ctypes.c_int32, ctypes.c_int32, P, P, P, P, P, ctypes.c_int64,
                                             P, ctypes.c_int64, P, P, ctypes.c_int64, P, ctypes.c_int32]
        L.oracle_run_batch_share.restype = ctypes.c_int
        L.oracle_critical_path.argtypes = [ctypes.c_int32, P, P, ctypes.c_int64, P, ctypes.c_int64,
                                           P, ctypes.c_int64, P, ctypes.c_int32, P, ctypes.c_int32]
        L.oracle_critical_path.restype = ctypes.c_int
        L.oracle_static_run.argtypes = [ctypes.c_int32, ctypes.c_int32, P, P, P, P, ctypes.c_int64,
                                        P, ctypes.c_int64, P, P, ctypes.c_int64, P, ctypes.c_int32]
        L.oracle_static_run.restype = ctypes.c_int
        L.oracle_attribute.argtypes = [ctypes.c_int32, ctypes.c_int32, P, P, P, P, ctypes.c_int64, P,
                                       ctypes.c_int64, P, ctypes.c_int64, P, P, P, P, ctypes.c_int64, P,
                                       ctypes.c_int64, P, ctypes.c_int32, P, ctypes.c_int32]
        L.oracle_attribute.restype = ctypes.c_int
        L.oracle_philox4x32_10.argtypes = [P, P, P]
        L.oracle_philox4x32_10.restype = None
        L.oracle_philox4x64_10.argtypes = [P, P, P]
        L.oracle_philox4x64_10.restype = None
        L.oracle_generate.argtypes = [ctypes.c_int32, ctypes.c_int64, P, ctypes.c_int32, ctypes.c_int64,
                                      ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int64, P, ctypes.c_int64,
                                      ctypes.c_int32]
        L.oracle_generate.restype = ctypes.c_int
        if path is not None:
            return L
        _lib = L
    return _lib


class OracleError(RuntimeError):
    def __init__(self, code: int):
        super().__init__(f"oracle error {code}")
        self.code = code


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


def _c(a, dt):
    return None if a is None else np.ascontiguousarray(a, dtype=dt)


def _threads(n_threads: Optional[int]) -> int:
    return n_threads if n_threads else len(os.sched_getaffinity(0))


def run_batch(succ_ptr, succ_idx, op_res, n_res: int, dur, prio=None, place=None,
              want_finish: bool = True, n_threads: Optional[int] = None, library=None, gap=None,
              delay=None):
    """Replay every scenario column of ``dur`` ([n_ops, n_scen] int32);
    ``gap`` ([n_res] int32 or None) is each device's idle time between
    consecutive ops, ``delay`` ([n_res] int32 or None) the time after an op
    finishes until its outputs reach its successors.

    Returns ``(makespan [S], finish [n_ops, S] or None, status [S])``.
    """
    succ_ptr, succ_idx = _c(succ_ptr, np.int64), _c(succ_idx, np.int32)
    op_res, prio, gap = _c(op_res, np.int32), _c(prio, np.int32), _c(gap, np.int32)
    delay = _c(delay, np.int32)
    dur, place = _c(dur, np.int32), _c(place, np.uint16)
    n = op_res.size
    S = dur.shape[1] if dur.ndim == 2 else 0
    makespan = np.empty(S, np.int32)
    status = np.empty(S, np.int32)
    finish = np.empty((n, S), np.int32) if want_finish else None
    L = library or lib()
    if delay is not None:
        rc = L.oracle_run_batch_dev(n, n_res, _ptr(succ_ptr), _ptr(succ_idx), _ptr(op_res), _ptr(prio),
                                    _ptr(gap), _ptr(delay), S, _ptr(dur), S, _ptr(place), S, _ptr(makespan),
                                    _ptr(finish), S, _ptr(status), _threads(n_threads))
    elif gap is None:
        rc = L.oracle_run_batch(n, n_res, _ptr(succ_ptr), _ptr(succ_idx), _ptr(op_res), _ptr(prio),
                                S, _ptr(dur), S, _ptr(place), S, _ptr(makespan), _ptr(finish), S,
                                _ptr(status), _threads(n_threads))
    else:
        rc = L.oracle_run_batch_gap(n, n_res, _ptr(succ_ptr), _ptr(succ_idx), _ptr(op_res), _ptr(prio),
                                    _ptr(gap), S, _ptr(dur), S, _ptr(place), S, _ptr(makespan), _ptr(finish),
                                    S, _ptr(status), _threads(n_threads))
    if rc:
        raise OracleError(rc)
    return makespan, finish, status


def run_batch_share(succ_ptr, succ_idx, op_res, n_res: int, dur, share=None, prio=None,
                    want_finish: bool = True, n_threads: Optional[int] = None, library=None):
    """Replay every scenario column of ``dur`` with bandwidth sharing on the
    devices where ``share`` ([n_res], nonzero: shared) is set.

    Returns ``(makespan [S], finish [n_ops, S] or None, status [S])``.
    """
    succ_ptr, succ_idx = _c(succ_ptr, np.int64), _c(succ_idx, np.int32)
    op_res, prio, dur = _c(op_res, np.int32), _c(prio, np.int32), _c(dur, np.int32)
    share = None if share is None else np.ascontiguousarray(np.asarray(share) != 0, dtype=np.uint8)
    n = op_res.size
    S = dur.shape[1] if dur.ndim == 2 else 0
    makespan = np.empty(S, np.int32)
    status = np.empty(S, np.int32)
    finish = np.empty((n, S), np.int32) if want_finish else None
    L = library or lib()
    rc = L.oracle_run_batch_share(n, n_res, _ptr(succ_ptr), _ptr(succ_idx), _ptr(op_res), _ptr(prio), _ptr(share),
                                  S, _ptr(dur), S, _ptr(makespan), _ptr(finish), S, _ptr(status),
                                  _threads(n_threads))
    if rc:
        raise OracleError(rc)
    return makespan, finish, status


def critical_path(succ_ptr, succ_idx, n_ops: int, dur, path_scen: int = -1,
                  n_threads: Optional[int] = None, library=None):
    """Longest path per scenario; returns ``(cp_len [S], path or None)``."""
    succ_ptr, succ_idx, dur = _c(succ_ptr, np.int64), _c(succ_idx, np.int32), _c(dur, np.int32)
    S = dur.shape[1] if dur.ndim == 2 else 0
    cp = np.empty(S, np.int32)
    cap = max(n_ops, 1)
    path = np.empty(cap, np.int32)
    plen = np.zeros(1, np.int32)
    rc = (library or lib()).oracle_critical_path(n_ops, _ptr(succ_ptr), _ptr(succ_idx), S, _ptr(dur), S,
                                    _ptr(cp), path_scen, _ptr(path), cap, _ptr(plen),
                                    _threads(n_threads))
    if rc:
        raise OracleError(rc)
    return cp, (path[: int(plen[0])].copy() if path_scen >= 0 else None)


def static_run(succ_ptr, succ_idx, op_res, n_res: int, order, dur, want_finish: bool = True,
               n_threads: Optional[int] = None, library=None):
    """Static-order replay of every scenario column of ``dur``: each device
    runs its ops in the order they appear in ``order``.  Returns
    ``(makespan [S], finish [n_ops, S] or None, status [S])``."""
    succ_ptr, succ_idx = _c(succ_ptr, np.int64), _c(succ_idx, np.int32)
    op_res, order, dur = _c(op_res, np.int32), _c(order, np.int32), _c(dur, np.int32)
    n = op_res.size
    S = dur.shape[1] if dur.ndim == 2 else 0
    makespan = np.empty(S, np.int32)
    status = np.empty(S, np.int32)
    finish = np.empty((n, S), np.int32) if want_finish else None
    rc = (library or lib()).oracle_static_run(n, n_res, _ptr(succ_ptr), _ptr(succ_idx), _ptr(op_res),
                                              _ptr(order), S, _ptr(dur), S, _ptr(makespan), _ptr(finish),
                                              S, _ptr(status), _threads(n_threads))
    if rc:
        raise OracleError(rc)
    return makespan, finish, status


def attribute(succ_ptr, succ_idx, op_res, n_res: int, dur, prio=None, place=None, path_scen: int = -1,
              n_threads: Optional[int] = None, library=None):
    """Bottleneck attribution of the replay of every scenario column of ``dur``.

    Returns ``(makespan [S], status [S], busy [n_res, S], chain [n_res, S],
    chain_ops [S], path or None)``: per resource its busy time and the time
    the binding chain spends on it, the chain's op count, and (for
    ``path_scen``) the chain from its first op to its last.
    """
    succ_ptr, succ_idx = _c(succ_ptr, np.int64), _c(succ_idx, np.int32)
    op_res, prio = _c(op_res, np.int32), _c(prio, np.int32)
    dur, place = _c(dur, np.int32), _c(place, np.uint16)
    n = op_res.size
    S = dur.shape[1] if dur.ndim == 2 else 0
    makespan = np.empty(S, np.int32)
    status = np.empty(S, np.int32)
    busy = np.empty((n_res, S), np.int32)
    chain = np.empty((n_res, S), np.int32)
    chain_ops = np.empty(S, np.int32)
    cap = max(n, 1)
    path = np.empty(cap, np.int32)
    plen = np.zeros(1, np.int32)
    rc = (library or lib()).oracle_attribute(n, n_res, _ptr(succ_ptr), _ptr(succ_idx), _ptr(op_res),
                                             _ptr(prio), S, _ptr(dur), S, _ptr(place), S, _ptr(makespan),
                                             _ptr(status), _ptr(busy), _ptr(chain), S, _ptr(chain_ops),
                                             path_scen, _ptr(path), cap, _ptr(plen), _threads(n_threads))
    if rc:
        raise OracleError(rc)
    return makespan, status, busy, chain, chain_ops, (path[: int(plen[0])].copy() if path_scen >= 0 else None)


def philox4x32_10(ctr, key, library=None) -> np.ndarray:
    """Philox4x32-10 of one counter block (4 uint32) under one key (2 uint32)."""
    c, k = np.asarray(ctr, np.uint32).copy(), np.asarray(key, np.uint32).copy()
    out = np.empty(4, np.uint32)
    (library or lib()).oracle_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def philox4x64_10(ctr, key, library=None) -> np.ndarray:
    """Philox4x64-10 of one counter block (4 uint64) under one key (2 uint64)."""
    c, k = np.asarray(ctr, np.uint64).copy(), np.asarray(key, np.uint64).copy()
    out = np.empty(4, np.uint64)
    (library or lib()).oracle_philox4x64_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def generate(base, n_scen: int, knob_block: int, noise: int, seed: int, scen0: int = 0,
             n_threads: Optional[int] = None, library=None) -> np.ndarray:
    """Generated durations int32 [n_ops, n_scen] from ``base`` ([n_knobs, n_ops]
    int32): knob grid times counter-based noise (``oracle.h`` states the formula)."""
    base = _c(np.atleast_2d(base), np.int32)
    n_knobs, n = base.shape
    dur = np.empty((n, n_scen), np.int32)
    rc = (library or lib()).oracle_generate(n, n_scen, _ptr(base), n_knobs, knob_block, noise,
                                            seed & (2**64 - 1), scen0, _ptr(dur), n_scen,
                                            _threads(n_threads))
    if rc:
        raise OracleError(rc)
    return dur
