"""Discrete-event simulation of a 1F1B pipeline (test infrastructure).

An independent second model of the same training iteration, used only to
pin the DAG oracle: S workers each run their own 1F1B task list in order;
a forward task on stage s > 1 may start only once the activation of the
same micro-batch has arrived from stage s - 1 (sent when that task ends,
arriving comm_fwd[s-2] later); a backward task on stage s < S waits for the
gradient from stage s + 1 (arriving comm_bwd[s-1] after it ends).  Each
worker starts a task as soon as it is idle and the task's input is there.
The iteration ends when the last worker finishes (Sec. 2.3: the iteration
time is set by the longest chain of such dependencies; Sec. 4.1 models the
same dependencies as DAG edges).

Nothing here builds a graph or takes a longest path: time advances through
an event queue, which is what makes it a separate check of the DAG.
"""
from __future__ import annotations

import heapq
from typing import Sequence


def simulate_1f1b(S: int, M: int, F: Sequence[int], B: Sequence[int],
                  cf: Sequence[int], cb: Sequence[int], order, allreduce=None) -> int:
    """Iteration time of the event-driven run; `order(S, M, s)` gives stage
    s's task list as ('F'|'B', m) pairs.  With `allreduce`, stage s starts
    its gradient all-reduce (allreduce[s-1] long) once its task list is done,
    and the iteration ends when the last all-reduce ends."""
    tasks = {s: order(S, M, s) for s in range(1, S + 1)}
    nxt = {s: 0 for s in tasks}
    busy_until = {s: 0 for s in tasks}
    idle = {s: True for s in tasks}
    arrived = set()          # (kind, stage, m): input of that task is present
    events = []              # (time, seq, kind, payload)
    seq = 0

    def push(t, kind, payload):
        nonlocal seq
        heapq.heappush(events, (t, seq, kind, payload))
        seq += 1

    def input_ready(s, kind, m):
        if kind == "F":
            return s == 1 or ("F", s, m) in arrived
        return s == S or ("B", s, m) in arrived

    def try_start(s, now):
        if not idle[s] or nxt[s] >= len(tasks[s]):
            return
        kind, m = tasks[s][nxt[s]]
        if not input_ready(s, kind, m):
            return
        dur = F[s - 1] if kind == "F" else B[s - 1]
        idle[s] = False
        push(now + dur, "done", (s, kind, m))

    end = 0
    for s in range(1, S + 1):
        try_start(s, 0)
    while events:
        now, _, ev, payload = heapq.heappop(events)
        end = max(end, now)
        if ev == "done":
            s, kind, m = payload
            idle[s] = True
            busy_until[s] = now
            nxt[s] += 1
            if kind == "F" and s < S:
                push(now + cf[s - 1], "arrive", ("F", s + 1, m))
            if kind == "B" and s > 1:
                push(now + cb[s - 2], "arrive", ("B", s - 1, m))
            try_start(s, now)
        else:
            arrived.add(payload)
            try_start(payload[1], now)
    if any(nxt[s] != len(tasks[s]) for s in tasks):
        raise RuntimeError("pipeline deadlocked")
    if allreduce is not None:
        return max(busy_until[s] + int(allreduce[s - 1]) for s in tasks)
    return max(busy_until.values()) if busy_until else end


def all_paths_longest(dag, F, B, cf, cb, d=None) -> int:
    """Brute force: enumerate every start->end path of the explicit DAG by
    depth-first search and take the largest node+edge weight sum (the
    definition of the critical path, App. B.1).  Exponential; tiny DAGs only."""
    succ = {}
    for u, v, k in dag.edges:
        succ.setdefault(u, []).append((v, k))

    def wnode(v):
        kind, s, _ = v
        if kind == "F":
            return F[s - 1]
        if kind == "B":
            return B[s - 1]
        if kind == "R":
            return d[s - 1] if d is not None else 0
        return 0

    def wedge(u, v, k):
        if k == "fwd":
            return cf[u[1] - 1]
        if k == "bwd":
            return cb[v[1] - 1]
        return 0

    best = -1
    stack = [(("S", 0, 0), 0)]
    while stack:
        u, acc = stack.pop()
        acc += wnode(u)
        if u == ("E", 0, 0):
            best = max(best, acc)
            continue
        for v, k in succ.get(u, []):
            stack.append((v, acc + wedge(u, v, k)))
    return best


def simulate_devices(S: int, N: int, M: int, F: Sequence[int], B: Sequence[int],
                     cf: Sequence[int], cb: Sequence[int], tasks, allreduce=None) -> int:
    """Event-driven run of a pipeline whose N devices hold several of the S
    virtual stages (Interleaved 1F1B): `tasks[p]` (p = 1..N) is device p's
    list of ('F'|'B', virtual stage j, m).  F on stage j > 1 waits for the
    activation of F_{j-1,m} (cf[j-2] after it ends); B on j < S waits for the
    gradient of B_{j+1,m} (cb[j-1] after it ends).  With `allreduce` (per
    device) each device then runs its all-reduce; the iteration ends with
    the last device."""
    nxt = {p: 0 for p in tasks}
    busy_until = {p: 0 for p in tasks}
    idle = {p: True for p in tasks}
    arrived = set()
    events = []
    seq = 0

    def push(t, kind, payload):
        nonlocal seq
        heapq.heappush(events, (t, seq, kind, payload))
        seq += 1

    def try_start(p, now):
        if not idle[p] or nxt[p] >= len(tasks[p]):
            return
        kind, j, m = tasks[p][nxt[p]]
        if kind == "F" and j > 1 and ("F", j, m) not in arrived:
            return
        if kind == "B" and j < S and ("B", j, m) not in arrived:
            return
        idle[p] = False
        push(now + (F[j - 1] if kind == "F" else B[j - 1]), "done", (p, kind, j, m))

    dev_of = {}
    for p, lst in tasks.items():
        for kind, j, m in lst:
            dev_of[j] = p
    for p in tasks:
        try_start(p, 0)
    while events:
        now, _, ev, payload = heapq.heappop(events)
        if ev == "done":
            p, kind, j, m = payload
            idle[p] = True
            busy_until[p] = now
            nxt[p] += 1
            if kind == "F" and j < S:
                push(now + cf[j - 1], "arrive", ("F", j + 1, m))
            if kind == "B" and j > 1:
                push(now + cb[j - 2], "arrive", ("B", j - 1, m))
            try_start(p, now)
        else:
            arrived.add(payload)
            try_start(dev_of[payload[1]], now)
    if any(nxt[p] != len(tasks[p]) for p in tasks):
        raise RuntimeError("pipeline deadlocked")
    if allreduce is not None:
        return max(busy_until[p] + int(allreduce[p - 1]) for p in tasks)
    return max(busy_until.values())
