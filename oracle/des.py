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
