"""Independent brute-force replays used to pin the CPU oracle.

Neither shares code with the oracle (which is C): they restate the paper's
simulation loop (Sec. 2, "Dataflow based simulation") in two other ways.

``tick_sim`` advances time one nanosecond at a time.  At each tick it first
retires every op that finishes at that tick (decrementing its successors'
dependency counters and appending newly ready ops to their device's job
queue), then every idle device starts the op at the head of its queue.  Ops
that become ready at the same tick enter a queue in (priority, id) order.

``enumerate_orders`` tries every per-device order of the ops, computes the
start times that order implies (an op starts when its predecessors and the
previous op on its device have finished), and keeps the orders in which every
device's sequence is sorted by (ready time, priority, id), i.e. a
first-in-first-out queue by ready time.
"""
from __future__ import annotations

import itertools
from collections import deque

import numpy as np


def preds_of(n, succ_ptr, succ_idx):
    P = [set() for _ in range(n)]
    for u in range(n):
        for e in range(int(succ_ptr[u]), int(succ_ptr[u + 1])):
            P[int(succ_idx[e])].add(u)
    return P


def tick_sim(n, n_res, succ_ptr, succ_idx, res, dur, prio=None, gap=None, delay=None):
    """One scenario: returns finish times (list) by 1-ns time stepping.

    With ``gap``, a device that finishes an op at t stays idle until
    t + gap[device] before it starts its next one.  With ``delay``, an op
    finishing at t on a device counts as done for its successors at
    t + delay[device].
    """
    prio = list(range(n)) if prio is None else [int(x) for x in prio]
    P = preds_of(n, succ_ptr, succ_idx)
    S = [set() for _ in range(n)]
    for v in range(n):
        for u in P[v]:
            S[u].add(v)
    cnt = [len(P[v]) for v in range(n)]
    queue = [deque() for _ in range(n_res)]
    running = [None] * n_res  # (op, finish)
    avail = [0] * n_res  # first tick at which each device may start an op
    arrive = {}  # tick -> ops whose outputs reach their successors then
    finish = [None] * n
    done = 0
    arrivals = sorted((v for v in range(n) if cnt[v] == 0), key=lambda v: (prio[v], v))
    for v in arrivals:
        queue[int(res[v])].append(v)
    t = 0
    limit = int(np.sum(dur)) + 1 + (n * int(max(gap)) if gap is not None and len(gap) else 0)
    limit += n * int(max(delay)) if delay is not None and len(delay) else 0
    while done < n or arrive:
        # retire everything finishing now
        for r in range(n_res):
            if running[r] is not None and running[r][1] == t:
                v = running[r][0]
                running[r] = None
                avail[r] = t + (int(gap[r]) if gap is not None else 0)
                done += 1
                arrive.setdefault(t + (int(delay[r]) if delay is not None else 0), []).append(v)
        # outputs arriving now count down their successors
        newly = []
        for v in arrive.pop(t, []):
            for w in S[v]:
                cnt[w] -= 1
                if cnt[w] == 0:
                    newly.append(w)
        for w in sorted(newly, key=lambda v: (prio[v], v)):
            queue[int(res[w])].append(w)
        # idle devices start their queue heads
        for r in range(n_res):
            if running[r] is None and queue[r] and t >= avail[r]:
                v = queue[r].popleft()
                finish[v] = t + int(dur[v])
                running[r] = (v, finish[v])
        t += 1
        if t > limit:
            raise RuntimeError("tick simulation did not terminate")
    return finish


def tick_sim_share(n, n_res, succ_ptr, succ_idx, res, dur, share, prio=None):
    """One scenario with bandwidth sharing, by 1-ns time stepping: finish
    times (list).

    A device with share[r] set runs every op ready on it at once; over each
    nanosecond its k active ops each receive 1/k ns of service (exact
    fractions), and an op leaves at the first tick at which its service
    reaches its duration.  Other devices run their queues first in first out
    as in tick_sim.
    """
    from fractions import Fraction
    prio = list(range(n)) if prio is None else [int(x) for x in prio]
    P = preds_of(n, succ_ptr, succ_idx)
    S = [set() for _ in range(n)]
    for v in range(n):
        for u in P[v]:
            S[u].add(v)
    cnt = [len(P[v]) for v in range(n)]
    queue = [deque() for _ in range(n_res)]
    running = [None] * n_res
    active = [dict() for _ in range(n_res)]  # shared devices: op -> service received
    finish = [None] * n

    def enter(ops):
        for v in sorted(ops, key=lambda v: (prio[v], v)):
            r = int(res[v])
            if share[r]:
                active[r][v] = Fraction(0)
            else:
                queue[r].append(v)

    enter([v for v in range(n) if cnt[v] == 0])
    done, t = 0, 0
    limit = int(np.sum(dur)) + n + 1
    while done < n:
        ended = []
        for r in range(n_res):
            if running[r] is not None and running[r][1] == t:
                ended.append(running[r][0])
                running[r] = None
            for v in [v for v, got in active[r].items() if got >= int(dur[v])]:
                del active[r][v]
                finish[v] = t
                ended.append(v)
        newly = []
        for v in ended:
            done += 1
            for w in S[v]:
                cnt[w] -= 1
                if cnt[w] == 0:
                    newly.append(w)
        enter(newly)
        for r in range(n_res):
            if running[r] is None and queue[r]:
                v = queue[r].popleft()
                finish[v] = t + int(dur[v])
                running[r] = (v, finish[v])
        for r in range(n_res):
            k = len(active[r])
            for v in active[r]:
                active[r][v] += Fraction(1, k)
        t += 1
        if t > limit:
            raise RuntimeError("tick simulation did not terminate")
    return finish


def _times_for_order(n, P, res, dur, orders, gap=None, delay=None):
    """Start/finish/ready times implied by per-device orders, or None if the
    orders contradict the DAG (a cycle through device and data edges)."""
    prev_on_dev = {}
    for seq in orders:
        for a, b in zip(seq, seq[1:]):
            prev_on_dev[b] = a
    finish = [None] * n
    ready = [None] * n
    remaining = set(range(n))
    while remaining:
        progress = False
        for v in sorted(remaining):
            if all(finish[u] is not None for u in P[v]) and (
                    v not in prev_on_dev or finish[prev_on_dev[v]] is not None):
                ready[v] = max([finish[u] + (int(delay[int(res[u])]) if delay is not None else 0)
                                for u in P[v]], default=0)
                avail = (finish[prev_on_dev[v]] + (int(gap[int(res[v])]) if gap is not None else 0)
                         if v in prev_on_dev else 0)
                start = max(ready[v], avail)
                finish[v] = start + int(dur[v])
                remaining.discard(v)
                progress = True
        if not progress:
            return None
    return ready, finish


def enumerate_orders(n, n_res, succ_ptr, succ_idx, res, dur, prio=None, gap=None, delay=None):
    """All per-device orders whose implied schedule is FIFO by (ready, prio, id).

    Returns a list of finish-time lists, one per consistent order.
    """
    prio = list(range(n)) if prio is None else [int(x) for x in prio]
    P = preds_of(n, succ_ptr, succ_idx)
    on = [[v for v in range(n) if int(res[v]) == r] for r in range(n_res)]
    found = []
    for orders in itertools.product(*[itertools.permutations(o) for o in on]):
        tr = _times_for_order(n, P, res, dur, orders, gap, delay)
        if tr is None:
            continue
        ready, finish = tr
        ok = all((ready[a], prio[a], a) < (ready[b], prio[b], b)
                 for seq in orders for a, b in zip(seq, seq[1:]))
        if ok:
            found.append(finish)
    return found


def all_path_lengths(n, succ_ptr, succ_idx, dur):
    """Longest path by enumerating every source-to-sink path (tiny DAGs)."""
    S = [[int(succ_idx[e]) for e in range(int(succ_ptr[u]), int(succ_ptr[u + 1]))] for u in range(n)]
    P = preds_of(n, succ_ptr, succ_idx)
    best = 0
    stack = [(v, int(dur[v])) for v in range(n) if not P[v]]
    while stack:
        v, L = stack.pop()
        best = max(best, L)
        for w in S[v]:
            stack.append((w, L + int(dur[w])))
    return best


def tick_sim_share_units(n, n_res, succ_ptr, succ_idx, res, dur, share, unit, prio=None):
    """One scenario with bandwidth sharing in whole service units, by 1-ns
    time stepping: finish times (list).

    A shared device delivers ``unit`` service units per ns.  Over each ns
    its k active ops each receive ``unit // k`` units (the share rounded
    down, so k ops that do not divide ``unit`` lose the remainder); an op of
    duration d leaves at the first tick at which it holds d * unit units.
    At a tick, every op that is done leaves (on shared and exclusive devices
    alike) before the ops it releases are entered, in (priority, id) order,
    and before idle exclusive devices start their queue heads; the newly
    entered ops share the next ns.  Written with plain integers and no
    event list, independently of the oracle's event-driven replay.
    """
    prio = list(range(n)) if prio is None else [int(x) for x in prio]
    P = preds_of(n, succ_ptr, succ_idx)
    S = [set() for _ in range(n)]
    for v in range(n):
        for u in P[v]:
            S[u].add(v)
    cnt = [len(P[v]) for v in range(n)]
    queue = [deque() for _ in range(n_res)]
    running = [None] * n_res
    held = [dict() for _ in range(n_res)]  # shared devices: op -> units received
    finish = [None] * n

    def enter(ops):
        for v in sorted(ops, key=lambda v: (prio[v], v)):
            r = int(res[v])
            if share[r]:
                held[r][v] = 0
            else:
                queue[r].append(v)

    enter([v for v in range(n) if cnt[v] == 0])
    done, t = 0, 0
    limit = int(np.sum(dur)) * 2 + n + 1
    while done < n:
        ended = []
        for r in range(n_res):
            if running[r] is not None and running[r][1] == t:
                ended.append(running[r][0])
                running[r] = None
            for v in [v for v, got in held[r].items() if got >= int(dur[v]) * unit]:
                del held[r][v]
                finish[v] = t
                ended.append(v)
        newly = []
        for v in ended:
            done += 1
            for w in S[v]:
                cnt[w] -= 1
                if cnt[w] == 0:
                    newly.append(w)
        enter(newly)
        for r in range(n_res):
            if running[r] is None and queue[r]:
                v = queue[r].popleft()
                finish[v] = t + int(dur[v])
                running[r] = (v, finish[v])
        for r in range(n_res):
            k = len(held[r])
            if k:
                per_op = unit // k
                for v in held[r]:
                    held[r][v] += per_op
        t += 1
        if t > limit:
            raise RuntimeError("tick simulation did not terminate")
    return finish
