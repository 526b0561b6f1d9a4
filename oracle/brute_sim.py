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


# ---------------------------------------------------------------------------
# Interleaved 1F1B (several model chunks per device, as in Megatron-LM):
# device s holds chunks j = 0..v-1, virtual stage j*S + s.


def interleaved_op_list(S, v, M, s):
    """Device s's ops as (kind, virtual stage, micro-batch), in the order it runs them:
    warm-up forwards, then one forward and one backward at a time, then the remaining
    backwards.  Forwards visit micro-batches in groups of S, chunk by chunk; backwards the
    same groups with the chunks in reverse."""
    n = M * v
    warm = min(n, 2 * (S - 1 - s) + (v - 1) * S)

    def fwd(k):
        g, r = divmod(k, S * v)
        return ("F", (r // S) * S + s, g * S + r % S)

    def bwd(k):
        g, r = divmod(k, S * v)
        return ("B", (v - 1 - r // S) * S + s, g * S + r % S)
    ops = [fwd(k) for k in range(warm)]
    for i in range(n - warm):
        ops.append(fwd(warm + i))
        ops.append(bwd(i))
    ops += [bwd(k) for k in range(n - warm, n)]
    return ops


def simulate_interleaved(S, v, M, f, b, c, cw):
    """Event-driven replay: f, b per virtual stage; c[s] the hop between devices s and s+1;
    cw the hop from the last device to the first (between chunks).  Returns the end time of
    each device's last op."""
    V = S * v
    lists = [interleaved_op_list(S, v, M, s) for s in range(S)]
    nxt = [0] * S
    busy = [False] * S
    idle_at = [0] * S
    arrived = set()                      # (kind, vs, m) inputs present at the device of vs
    for m in range(M):
        arrived.add(("F", 0, m))
    events = []
    seq = 0

    def push(t, kind, data):
        nonlocal seq
        heapq.heappush(events, (t, seq, kind, data))
        seq += 1

    def hop(vs_from, vs_to):
        """Forward hops go vs -> vs + 1, backward ones vs -> vs - 1; the one between the
        last device and the first (either way) is cw."""
        lo = min(vs_from, vs_to) % S
        return c[lo] if lo < S - 1 else cw

    def try_start(s, now):
        if busy[s] or nxt[s] >= len(lists[s]):
            return
        kind, vs, m = lists[s][nxt[s]]
        if (kind, vs, m) not in arrived:
            return
        busy[s] = True
        push(now + (f[vs] if kind == "F" else b[vs]), "done", (s, kind, vs, m))

    for s in range(S):
        try_start(s, 0)
    while events:
        now, _, kind, data = heapq.heappop(events)
        if kind == "done":
            s, k, vs, m = data
            busy[s] = False
            idle_at[s] = now
            nxt[s] += 1
            if k == "F":
                if vs + 1 < V:
                    push(now + hop(vs, vs + 1), "arrive", ("F", vs + 1, m))
                else:
                    arrived.add(("B", vs, m))
            elif vs > 0:
                push(now + hop(vs, vs - 1), "arrive", ("B", vs - 1, m))
            try_start(s, now)
        else:
            arrived.add(data)
            try_start(data[1] % S, now)
    for s in range(S):
        assert nxt[s] == len(lists[s]), "simulation stalled"
    return idle_at


# ---------------------------------------------------------------------------
# Zero-bubble order (ZB-H1, Qi et al. 2024): the backward pass splits into B
# (input gradient, sent upstream) and W (weight gradient, local).


def zb_op_list(S, M, s):
    """Stage s's ops: the 1F1B order of forwards and input-gradient passes, with each weight-
    gradient pass queued behind its B and released s micro-batches later; the queue empties
    at the end."""
    warm = min(S - 1 - s, M)
    ops = [("F", m) for m in range(warm)]
    queue = []
    f_next = warm
    for i in range(M):
        if f_next < M:
            ops.append(("F", f_next))
            f_next += 1
        ops.append(("B", i))
        queue.append(i)
        if len(queue) > s:
            ops.append(("W", queue.pop(0)))
    ops += [("W", m) for m in queue]
    return ops


def simulate_zb(S, M, f, bi, w, c):
    """Event-driven replay; f, bi, w per stage, c[s] the hop between stages s and s+1.  Returns
    the end time of each stage's last op."""
    lists = [zb_op_list(S, M, s) for s in range(S)]
    nxt = [0] * S
    busy = [False] * S
    idle_at = [0] * S
    arrived = {("F", 0, m) for m in range(M)}
    events = []
    seq = 0

    def push(t, kind, data):
        nonlocal seq
        heapq.heappush(events, (t, seq, kind, data))
        seq += 1

    def try_start(s, now):
        if busy[s] or nxt[s] >= len(lists[s]):
            return
        kind, m = lists[s][nxt[s]]
        if kind != "W" and (kind, s, m) not in arrived:
            return
        busy[s] = True
        push(now + {"F": f, "B": bi, "W": w}[kind][s], "done", (s, kind, m))

    for s in range(S):
        try_start(s, 0)
    while events:
        now, _, kind, data = heapq.heappop(events)
        if kind == "done":
            s, k, m = data
            busy[s] = False
            idle_at[s] = now
            nxt[s] += 1
            if k == "F":
                if s + 1 < S:
                    push(now + c[s], "arrive", ("F", s + 1, m))
                else:
                    arrived.add(("B", s, m))
            elif k == "B" and s > 0:
                push(now + c[s - 1], "arrive", ("B", s - 1, m))
            try_start(s, now)
        else:
            arrived.add(data)
            try_start(data[1], now)
    for s in range(S):
        assert nxt[s] == len(lists[s]), "simulation stalled"
    return idle_at
