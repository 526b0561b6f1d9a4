"""Brute-force discrete-event simulation of one 1F1B pipeline (tiny inputs only).

TEST INFRASTRUCTURE ONLY.  An independent check of the pipeline recurrence in
oracle.c: instead of sweeping a dependency graph it replays the training step
as a time-ordered event queue, the way an event-driven simulator does (Sec. 4.2
"System layer": an event queue and a scheduler that honours dependencies).

Model: each stage is a worker that executes its fixed 1F1B op list one op at a
time (non-interleaved schedule: forwards to fill the pipeline, then one forward
one backward, then the remaining backwards).  Finishing F(s, m) sends an
activation that reaches stage s+1 after c[s]; finishing B(s, m) sends a gradient
that reaches stage s-1 after c[s-1].  Sending never blocks the sender.  An op
starts at the first event time at which its worker is idle and its input is
present.
"""
import heapq


def op_list(S, M, s):
    W = min(S - 1 - s, M)
    ops = [("F", m) for m in range(W)]
    for i in range(M - W):
        ops.append(("F", W + i))
        ops.append(("B", i))
    ops += [("B", m) for m in range(M - W, M)]
    return ops


def simulate(S, M, f, b, c):
    """Return (end time of each stage's last op, [(stage, op, start, end)])."""
    lists = [op_list(S, M, s) for s in range(S)]
    nxt = [0] * S
    busy = [False] * S
    idle_at = [0] * S
    arrived = set()              # ("F", s, m): activation of micro-batch m present at stage s
    for m in range(M):
        arrived.add(("F", 0, m))  # stage 0 reads its input locally
    events = []                   # (time, seq, kind, data)
    seq = 0
    trace = []

    def push(t, kind, data):
        nonlocal seq
        heapq.heappush(events, (t, seq, kind, data))
        seq += 1

    def try_start(s, now):
        if busy[s] or nxt[s] >= len(lists[s]):
            return
        kind, m = lists[s][nxt[s]]
        if (kind, s, m) not in arrived:
            return
        busy[s] = True
        dur = f[s] if kind == "F" else b[s]
        push(now + dur, "done", (s, kind, m, now))

    now = 0
    for s in range(S):
        try_start(s, now)
    while events:
        now, _, kind, data = heapq.heappop(events)
        if kind == "done":
            s, k, m, start = data
            trace.append((s, k + str(m), start, now))
            busy[s] = False
            idle_at[s] = now
            nxt[s] += 1
            if k == "F":
                if s + 1 < S:
                    push(now + c[s], "arrive", ("F", s + 1, m))
                else:
                    arrived.add(("B", s, m))      # the loss is computed where the forward ended
            else:
                if s > 0:
                    push(now + c[s - 1], "arrive", ("B", s - 1, m))
            try_start(s, now)
            if k == "F" and s + 1 == S:
                try_start(s, now)
        else:
            arrived.add(data)
            try_start(data[1], now)
    for s in range(S):
        assert nxt[s] == len(lists[s]), "simulation stalled"
    return idle_at, trace
